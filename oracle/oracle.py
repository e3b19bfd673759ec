"""fp64 CPU oracle for the selective-SSM primal + tangent (JVP) scan.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the benchmark's CPU-baseline leg, never by the product path.  It shares no
code with the HIP path; both consume arrays from the seeded input module.

Layers
------
* ``core``: the per-lane recurrence of Lemma 3.1 (Eq. 3) and the output map,
  given explicit per-step coefficients (C, fp64, in ``pgf_oracle.c``).
* ``discretize``: Delta = softplus(x*w_delta + b_delta) and its tangent
  dDelta_k = sigmoid(z)*w_delta*dx_k (softplus' = sigmoid), per (b,t,d).  The
  selective step size follows the Mamba parameterisation the paper studies
  (Sec. 3; Lemma 3.1 makes Delta a function of the input).
* ``project``: B_t = x_t W_B (+ b_B), C_t = x_t W_C (+ b_C) and their tangents
  dB_k = dx_k W_B, dC_k = dx_k W_C (selective input/output maps, Sec. 3).
* ``scan_jvp``: the three above over L-chunks with the state carried between
  chunks (the block hand-off of Alg. 1), optionally for a subset of channels.
* ``core2`` / ``discretize2`` / ``scan_jvp2``: the second-order flow of
  App. G (mixed second directional derivative along two input directions
  v, w, with both first-order flows), same layering.
* ``core_param`` / ``param_grads``: the parameter-sensitivity flows and the
  online gradient accumulation of App. E (Alg. 2) for a given adjoint
  signal dl/dy, same layering.
* ``la_scan_jvp``: decaying linear attention (App. F: RetNet, RWKV-6,
  linear transformers) with its tangent flow, over L-chunks.

Precision: everything in fp64 from the exact fp32 / bf16 input values.
Library routines used as steps: numpy.logaddexp (softplus), scipy expit
(sigmoid), numpy matmul (projections), libm exp (transition).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
from scipy.special import expit

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pgf_oracle.c")
_DEFAULT_LIB = os.path.join(_HERE, "liboracle.so")
# PGF_ORACLE_LIB selects another build of the same source (the sanitized
# build of the tests).
_LIB_PATH = os.environ.get("PGF_ORACLE_LIB") or _DEFAULT_LIB
_lib = None
FLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra"]


def build(verbose: bool = False, out: str | None = None, extra: tuple = ()) -> str:
    """Compile the C core into oracle/liboracle.so, or `out` with `extra`
    compiler flags appended (always recompiles)."""
    out = out or _DEFAULT_LIB
    cmd = ["gcc", *FLAGS, *extra, "-o", out + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def declare(lib):
    """Declares the C signatures on a loaded oracle library (also used by
    the tests that load mutated copies of it)."""
    dp = ctypes.POINTER(ctypes.c_double)
    i64 = ctypes.c_int64
    lib.pgf_oracle_core.restype = ctypes.c_int
    lib.pgf_oracle_core.argtypes = [i64] * 5 + [dp] * 13 + [ctypes.c_int, ctypes.c_int]
    lib.pgf_oracle_core2.restype = ctypes.c_int
    lib.pgf_oracle_core2.argtypes = [i64] * 4 + [dp] * 22 + [ctypes.c_int]
    lib.pgf_oracle_param.restype = ctypes.c_int
    lib.pgf_oracle_param.argtypes = [i64] * 4 + [dp] * 14 + [ctypes.c_int] + [dp] * 8 + [ctypes.c_int, ctypes.c_int]
    lib.pgf_oracle_la.restype = ctypes.c_int
    lib.pgf_oracle_la.argtypes = [i64] * 6 + [dp] * 12 + [ctypes.c_int]
    lib.pgf_oracle_core_cplx.restype = ctypes.c_int
    lib.pgf_oracle_core_cplx.argtypes = [i64] * 5 + [dp] * 16 + [ctypes.c_int, ctypes.c_int]
    return lib


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    _lib = declare(ctypes.CDLL(_LIB_PATH))
    return _lib


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _threads() -> int:
    return int(os.environ.get("PGF_ORACLE_THREADS", "0"))


DRIVES = {"euler": 0, "zoh": 1}


def core(A, x, dx, delta, ddelta, Bm, Cm, dBm, dCm, h=None, dh=None, nthreads=None, drive="euler"):
    """Run the recurrence.  Shapes: A [D,N]; x, delta [B,L,D]; dx, ddelta
    [K,B,L,D]; Bm, Cm [B,L,N]; dBm, dCm [K,B,L,N]; h [B,D,N]; dh [K,B,D,N].
    drive: "euler" (Delta*B*x) or "zoh" (A^-1 (Abar - 1) B x).
    Returns (y [B,L,D], dy [K,B,L,D], h_out, dh_out), all fp64; y and dy
    are the state read-out sum_n C h (before any activation)."""
    lib = _load()
    A = _f64(A)
    x, dx, delta, ddelta = _f64(x), _f64(dx), _f64(delta), _f64(ddelta)
    Bm, Cm, dBm, dCm = _f64(Bm), _f64(Cm), _f64(dBm), _f64(dCm)
    K, B, L, D = dx.shape
    N = A.shape[1]
    assert A.shape == (D, N) and x.shape == (B, L, D) and delta.shape == (B, L, D)
    assert ddelta.shape == (K, B, L, D) and Bm.shape == (B, L, N) and Cm.shape == (B, L, N)
    assert dBm.shape == (K, B, L, N) and dCm.shape == (K, B, L, N)
    h = np.zeros((B, D, N)) if h is None else np.array(h, dtype=np.float64, copy=True, order="C")
    dh = np.zeros((K, B, D, N)) if dh is None else np.array(dh, dtype=np.float64, copy=True, order="C")
    assert h.shape == (B, D, N) and dh.shape == (K, B, D, N)
    y = np.empty((B, L, D))
    dy = np.empty((K, B, L, D))
    rc = lib.pgf_oracle_core(B, L, D, N, K, _dp(A), _dp(x), _dp(dx), _dp(delta), _dp(ddelta),
                             _dp(Bm), _dp(Cm), _dp(dBm), _dp(dCm), _dp(h), _dp(dh), _dp(y), _dp(dy),
                             DRIVES[drive], _threads() if nthreads is None else nthreads)
    if rc != 0:
        raise RuntimeError("pgf_oracle_core failed")
    return y, dy, h, dh


def discretize(x, dx, w_delta, b_delta):
    """Delta = softplus(z), dDelta_k = sigmoid(z) * w_delta * dx_k with
    z = x*w_delta + b_delta, per (b,t,d).  x [B,L,D], dx [K,B,L,D]."""
    x = _f64(x)
    w = _f64(w_delta)
    z = x * w + _f64(b_delta)
    delta = np.logaddexp(0.0, z)
    sw = expit(z) * w
    ddelta = sw[None] * _f64(dx)
    return delta, ddelta


def discretize_lowrank(x, dx, W_dx, W_dt, b_dt):
    """Mamba's low-rank step size: z = (x W_dx) W_dt + b_dt with W_dx [D,R],
    W_dt [R,D] (the rank-R bottleneck over all channels), Delta =
    softplus(z), dDelta_k = sigmoid(z) * ((dx_k W_dx) W_dt).
    x [B,L,D], dx [K,B,L,D] -> Delta [B,L,D], dDelta [K,B,L,D]."""
    x, dx = _f64(x), _f64(dx)
    Wx, Wt = _f64(W_dx), _f64(W_dt)
    z = (x @ Wx) @ Wt + _f64(b_dt)
    dz = (dx @ Wx) @ Wt
    return np.logaddexp(0.0, z), expit(z)[None] * dz


def project(x, dx, W_B, W_C, b_B=None, b_C=None):
    """B = x W_B (+b_B), C = x W_C (+b_C), dB_k = dx_k W_B, dC_k = dx_k W_C.
    x [B,L,D] -> [B,L,N]; dx [K,B,L,D] -> [K,B,L,N]."""
    x, dx = _f64(x), _f64(dx)
    WB, WC = _f64(W_B), _f64(W_C)
    Bm = x @ WB
    Cm = x @ WC
    if b_B is not None:
        Bm = Bm + _f64(b_B)
    if b_C is not None:
        Cm = Cm + _f64(b_C)
    return Bm, Cm, dx @ WB, dx @ WC


def core_cplx(A, Aim, x, dx, delta, ddelta, Bm, Cm, dBm, dCm, h=None, dh=None, nthreads=None, drive="euler"):
    """The recurrence with a complex diagonal transition A + i*Aim (see
    pgf_oracle_core_cplx), Euler or zero-order-hold drive.  h [B,D,N] and
    dh [K,B,D,N] are complex (zero when None).  Returns (y, dy, h_out,
    dh_out); y and dy are the real read-out sum_n C Re(h)."""
    lib = _load()
    A, Aim = _f64(A), _f64(Aim)
    x, dx, delta, ddelta = _f64(x), _f64(dx), _f64(delta), _f64(ddelta)
    Bm, Cm, dBm, dCm = _f64(Bm), _f64(Cm), _f64(dBm), _f64(dCm)
    K, B, L, D = dx.shape
    N = A.shape[1]
    h = np.zeros((B, D, N), complex) if h is None else np.asarray(h, complex)
    dh = np.zeros((K, B, D, N), complex) if dh is None else np.asarray(dh, complex)
    parts = [np.ascontiguousarray(a, dtype=np.float64) for a in (h.real, h.imag, dh.real, dh.imag)]
    y = np.empty((B, L, D))
    dy = np.empty((K, B, L, D))
    rc = lib.pgf_oracle_core_cplx(B, L, D, N, K, _dp(A), _dp(Aim), _dp(x), _dp(dx), _dp(delta), _dp(ddelta),
                                  _dp(Bm), _dp(Cm), _dp(dBm), _dp(dCm), *[_dp(p) for p in parts], _dp(y), _dp(dy),
                                  DRIVES[drive], _threads() if nthreads is None else nthreads)
    if rc != 0:
        raise RuntimeError("pgf_oracle_core_cplx failed")
    return y, dy, parts[0] + 1j * parts[1], parts[2] + 1j * parts[3]


def channel_groups(channels, D, G):
    """Group of each channel: contiguous blocks of D/G channels."""
    return np.asarray(channels) // (D // G)


ACTIVATIONS = ("identity", "silu")


def output_map(yr, dyr, x, dx, D_res=None, act="identity"):
    """The output map of Sec. 3 applied to the state read-out yr = sum_n C h
    and its tangents dyr [K,...]: y_hat = yr + D_res*x, y = act(y_hat),
    dy_k = act'(y_hat) * (dyr_k + D_res*dx_k).  act: identity or SiLU
    (z*sigmoid(z), derivative s + z*s*(1-s))."""
    yh, dyh = _f64(yr), _f64(dyr)
    if D_res is not None:
        Dr = _f64(D_res)
        yh = yh + Dr * _f64(x)
        dyh = dyh + Dr * _f64(dx)
    if act == "identity":
        return yh, dyh
    if act == "silu":
        s = expit(yh)
        return yh * s, (s + yh * s * (1.0 - s))[None] * dyh
    raise ValueError(act)


def scan_jvp(x, dx, params, h_in=None, dh_in=None, channels=None, chunk=None, nthreads=None, drive="euler",
             act="identity"):
    """Full model: discretization, projections, recurrence, output map, over
    L-chunks.

    x [B,L,D], dx [K,B,L,D] (any float dtype; converted exactly to fp64).
    params: dict with A, w_delta, b_delta, W_B, W_C and optional b_B, b_C,
    D_res [D] (residual weight of the output map) and A_im [D,N] (the
    imaginary part of a complex diagonal transition: the state is complex,
    h_out/dh_out are returned complex, and y reads Re(C h)), and n_groups G
    (channel groups with their own B and C: W_B, W_C [D, G*N], b_B, b_C
    [G*N]; channel d uses group d // (D/G)), and W_dx [D,R], W_dt [R,D]
    (Mamba's low-rank step size, see discretize_lowrank; b_delta is its
    bias and w_delta is not used).
    drive: "euler" or "zoh" (the input drive, see core); act: "identity" or
    "silu" (the output activation, see output_map).
    channels: optional 1-D index array of channels d to compute (the
    projections still use every channel).  h_in [B,D,N] / dh_in [K,B,D,N]
    are over all D channels (or only the selected ones if shaped so).
    Returns (y [B,L,Dsel], dy [K,B,L,Dsel], h_out [B,Dsel,N], dh_out).
    """
    K, B, L, D = dx.shape
    A = _f64(params["A"])
    N = A.shape[1]
    sel = np.arange(D) if channels is None else np.asarray(channels, dtype=np.int64)
    Ds = len(sel)
    cplx = params.get("A_im") is not None
    cast = (lambda a: np.asarray(a, dtype=complex)) if cplx else _f64
    h = np.zeros((B, Ds, N)) if h_in is None else cast(h_in)
    dh = np.zeros((K, B, Ds, N)) if dh_in is None else cast(dh_in)
    if h.shape[1] == D and Ds != D:
        h = h[:, sel]
    if dh.shape[2] == D and Ds != D:
        dh = dh[:, :, sel]
    y = np.empty((B, L, Ds))
    dy = np.empty((K, B, L, Ds))
    step = L if not chunk else int(chunk)
    step = max(step, 1)
    lowrank = params.get("W_dt") is not None
    w = None if lowrank else _f64(params["w_delta"])[sel]
    bd = _f64(params["b_delta"])[sel]
    Dr = None if params.get("D_res") is None else _f64(params["D_res"])[sel]
    As = A[sel]
    G = int(params.get("n_groups") or 1)
    if D % G:
        raise ValueError("n_groups must divide the channel count")
    grp = channel_groups(sel, D, G)
    h = np.array(h, copy=True)
    dh = np.array(dh, copy=True)
    if cplx:
        Ais = _f64(params["A_im"])[sel]
        h = np.asarray(h, complex)
        dh = np.asarray(dh, complex)
    for t0 in range(0, L, step):
        t1 = min(L, t0 + step)
        xc = _f64(x[:, t0:t1])
        dxc = _f64(dx[:, :, t0:t1])
        Bm, Cm, dBm, dCm = project(xc, dxc, params["W_B"], params["W_C"],
                                   params.get("b_B"), params.get("b_C"))
        xs = np.ascontiguousarray(xc[..., sel])
        dxs = np.ascontiguousarray(dxc[..., sel])
        if lowrank:
            delta, ddelta = discretize_lowrank(xc, dxc, params["W_dx"], params["W_dt"], params["b_delta"])
            delta, ddelta = np.ascontiguousarray(delta[..., sel]), np.ascontiguousarray(ddelta[..., sel])
        else:
            delta, ddelta = discretize(xs, dxs, w, bd)
        # Channel groups: channel d reads the B, C of group d // (D / G)
        # (columns [g N, (g+1) N) of the projections); groups are independent
        # given their B and C, so each runs as its own recurrence.
        yc = np.empty((B, t1 - t0, Ds))
        dyc = np.empty((K, B, t1 - t0, Ds))
        for g in range(G):
            m = grp == g
            if not m.any():
                continue
            cols = slice(g * N, (g + 1) * N)
            args = (As[m], xs[..., m], dxs[..., m], delta[..., m], ddelta[..., m], Bm[..., cols], Cm[..., cols],
                    dBm[..., cols], dCm[..., cols], h[:, m], dh[:, :, m], nthreads)
            if cplx:
                yg, dyg, hg, dhg = core_cplx(args[0], Ais[m], *args[1:], drive=drive)
            else:
                yg, dyg, hg, dhg = core(*args, drive)
            yc[..., m], dyc[..., m] = yg, dyg
            h[:, m], dh[:, :, m] = hg, dhg
        y[:, t0:t1], dy[:, :, t0:t1] = output_map(yc, dyc, xs, dxs, Dr, act)
    return y, dy, h, dh


# ------------------------------------------------------------------ second order

def core2(A, x, xv, xw, delta, dv, dw, dvw, Bm, Cm, Bv, Cv, Bw, Cw, state=None, nthreads=None):
    """Second-order recurrence (see pgf_oracle_core2).  Shapes: A [D,N];
    x, xv, xw, delta, dv, dw, dvw [B,L,D]; Bm, Cm, Bv, Cv, Bw, Cw [B,L,N];
    state = (h, hv, hw, hvw), each [B,D,N] (zero when None).
    Returns (y, yv, yw, yvw) [B,L,D] and the exit state tuple."""
    lib = _load()
    A = _f64(A)
    arrs = [_f64(a) for a in (x, xv, xw, delta, dv, dw, dvw, Bm, Cm, Bv, Cv, Bw, Cw)]
    B, L, D = arrs[0].shape
    N = A.shape[1]
    for a in arrs[:7]:
        assert a.shape == (B, L, D)
    for a in arrs[7:]:
        assert a.shape == (B, L, N)
    if state is None:
        st = [np.zeros((B, D, N)) for _ in range(4)]
    else:
        st = [np.array(s, dtype=np.float64, copy=True, order="C") for s in state]
    for s_ in st:
        assert s_.shape == (B, D, N)
    outs = [np.empty((B, L, D)) for _ in range(4)]
    rc = lib.pgf_oracle_core2(B, L, D, N, _dp(A), *[_dp(a) for a in arrs], *[_dp(s_) for s_ in st],
                              *[_dp(o) for o in outs], _threads() if nthreads is None else nthreads)
    if rc != 0:
        raise RuntimeError("pgf_oracle_core2 failed")
    return tuple(outs), tuple(st)


def discretize2(x, xv, xw, w_delta, b_delta):
    """Delta = softplus(z) and its derivatives along v and w, z = x*w_delta
    + b_delta:  dv = s*w*xv, dw = s*w*xw, dvw = s*(1-s)*w^2*xv*xw with
    s = sigmoid(z) = softplus'(z) and s*(1-s) = softplus''(z)."""
    x = _f64(x)
    w = _f64(w_delta)
    z = x * w + _f64(b_delta)
    delta = np.logaddexp(0.0, z)
    s = expit(z)
    xv, xw = _f64(xv), _f64(xw)
    return delta, s * w * xv, s * w * xw, s * (1.0 - s) * w * w * xv * xw


def scan_jvp2(x, dxv, dxw, params, state=None, channels=None, chunk=None, nthreads=None):
    """Primal, both first-order flows and the mixed second-order flow of the
    full model over L-chunks.  x, dxv, dxw [B,L,D]; params as scan_jvp.
    Returns ((y, yv, yw, yvw) each [B,L,Dsel], exit state tuple)."""
    B, L, D = np.shape(x)
    A = _f64(params["A"])
    N = A.shape[1]
    sel = np.arange(D) if channels is None else np.asarray(channels, dtype=np.int64)
    Ds = len(sel)
    st = None if state is None else tuple(_f64(s_)[:, sel] if _f64(s_).shape[1] == D and Ds != D else _f64(s_)
                                          for s_ in state)
    outs = [np.empty((B, L, Ds)) for _ in range(4)]
    step = max(1, L if not chunk else int(chunk))
    w = _f64(params["w_delta"])[sel]
    bd = _f64(params["b_delta"])[sel]
    As = A[sel]
    for t0 in range(0, L, step):
        t1 = min(L, t0 + step)
        xc = _f64(x[:, t0:t1])
        vc = _f64(dxv[:, t0:t1])
        wc = _f64(dxw[:, t0:t1])
        Bm, Cm, dB, dC = project(xc, np.stack([vc, wc]), params["W_B"], params["W_C"],
                                 params.get("b_B"), params.get("b_C"))
        xs, vs, ws = (np.ascontiguousarray(a[..., sel]) for a in (xc, vc, wc))
        delta, dv, dw, dvw = discretize2(xs, vs, ws, w, bd)
        o, st = core2(As, xs, vs, ws, delta, dv, dw, dvw, Bm, Cm, dB[0], dC[0], dB[1], dC[1], st, nthreads)
        for i in range(4):
            outs[i][:, t0:t1] = o[i]
    return tuple(outs), st


# ------------------------------------------------------------------ parameter flows

ACTIVATIONS = {"identity": 0, "silu": 1}


def core_param(A, x, delta, gy, Bm, Cm, state=None, nthreads=None, drive="euler", act="identity", D_res=None,
               sig=None, scale=None):
    """Parameter-sensitivity flows (see pgf_oracle_param).  Shapes: A [D,N];
    x, delta, gy [B,L,D]; Bm, Cm [B,L,N]; state = (h, GammaA, GammaB), each
    [B,D,N] (zero when None); drive "euler" or "zoh" (the zero-order-hold
    drive, whose A-dependence enters GammaA); act "identity" or "silu" and
    D_res [D] or None: the output map y = act(sum_n C h + D_res x).
    sig [B,L,D] (sigmoid of the step size's pre-activation) adds the flows
    of w_delta and b_delta: the state tuple then has five entries (h,
    GammaA, GammaB, Gamma_w, Gamma_s).
    Returns y [B,L,D], (GA, GB, GC) each [B,D,N] (this call's contributions
    per batch row), plus GD [B,D] (dl/dD_res per batch row) when D_res is
    given, plus GW, GS [B,D] (dl/dw_delta, dl/db_delta) when sig is, and the
    exit state tuple.  scale: a pair of [B,D] arrays that receive (added to)
    the sums of the absolute values of the terms of GW and GS."""
    lib = _load()
    A = _f64(A)
    x, delta, gy, Bm, Cm = (_f64(a) for a in (x, delta, gy, Bm, Cm))
    B, L, D = x.shape
    N = A.shape[1]
    assert delta.shape == (B, L, D) and gy.shape == (B, L, D)
    assert Bm.shape == (B, L, N) and Cm.shape == (B, L, N)
    ns = 3 if sig is None else 5
    if state is None:
        st = [np.zeros((B, D, N)) for _ in range(ns)]
    else:
        st = [np.array(s, dtype=np.float64, copy=True, order="C") for s in state]
    assert len(st) == ns
    for s_ in st:
        assert s_.shape == (B, D, N)
    y = np.empty((B, L, D))
    G = [np.zeros((B, D, N)) for _ in range(3)]
    Dr = None if D_res is None else _f64(D_res)
    GD = None if D_res is None else np.zeros((B, D))
    null = ctypes.POINTER(ctypes.c_double)()
    sg = None if sig is None else _f64(sig)
    GWS = None if sig is None else [np.zeros((B, D)), np.zeros((B, D))]
    if sg is not None:
        assert sg.shape == (B, L, D)
    dres = [null if Dr is None else _dp(Dr), ACTIVATIONS[act], null if GD is None else _dp(GD)]
    dlt = [null] * 5 if sg is None else [_dp(sg), _dp(st[3]), _dp(st[4]), _dp(GWS[0]), _dp(GWS[1])]
    if scale is not None:
        assert sg is not None and all(a.shape == (B, D) and a.dtype == np.float64 for a in scale)
    dlt += [null, null] if scale is None else [_dp(scale[0]), _dp(scale[1])]
    rc = lib.pgf_oracle_param(B, L, D, N, _dp(A), _dp(x), _dp(delta), _dp(gy), _dp(Bm), _dp(Cm),
                              *[_dp(s_) for s_ in st[:3]], _dp(y), *[_dp(g) for g in G], *dres, *dlt,
                              DRIVES[drive], _threads() if nthreads is None else nthreads)
    if rc != 0:
        raise RuntimeError("pgf_oracle_param failed")
    if GD is not None:
        G.append(GD)
    if GWS is not None:
        G.extend(GWS)
    return y, tuple(G), tuple(st)


def param_grads(x, gy, params, state=None, chunk=None, channels=None, nthreads=None, drive="euler",
                act="identity", delta_params=False, return_scale=False):
    """Primal output and online parameter gradients of the full model over
    L-chunks (App. E, Alg. 2).  x, gy [B,L,D]; params as scan_jvp; channels:
    optional 1-D index array of the channels d to compute (the projections
    still use every channel; state and outputs cover only those).

    Returns (y [B,L,Dsel], (G_A, G_B, G_C) each [Dsel,N] summed over the
    batch, exit state (h, GammaA, GammaB) each [B,Dsel,N]).  drive: "euler"
    or "zoh" (see core_param).  G_A = dl/dA;
    G_B and G_C are the gradients with respect to per-lane offsets of B and
    C, so that dl/db_B = G_B.sum(0) and dl/db_C = G_C.sum(0).  act and
    params["D_res"] (if present) set the output map y = act(C h + D_res x);
    with D_res the gradient tuple gains G_D = dl/dD_res [Dsel].  With
    delta_params it then gains dl/dw_delta and dl/db_delta [Dsel] (the
    step size's parameters), and the state holds Gamma_w and Gamma_s after
    GammaB.  return_scale (with delta_params) appends the summation scales
    of those two gradients, sum over b and t of the absolute values of
    their terms [Dsel] each."""
    B, L, D = np.shape(x)
    A = _f64(params["A"])
    N = A.shape[1]
    sel = np.arange(D) if channels is None else np.asarray(channels, dtype=np.int64)
    Ds = len(sel)
    w = _f64(params["w_delta"])[sel]
    bd = _f64(params["b_delta"])[sel]
    As = A[sel]
    Dr = params.get("D_res")
    Dr = None if Dr is None else _f64(Dr)[sel]
    y = np.empty((B, L, Ds))
    tot = [np.zeros((B, Ds, N)) for _ in range(3)] + ([] if Dr is None else [np.zeros((B, Ds))]) + \
        ([np.zeros((B, Ds)), np.zeros((B, Ds))] if delta_params else [])
    scale = [np.zeros((B, Ds)), np.zeros((B, Ds))] if return_scale else None
    st = state
    step = max(1, L if not chunk else int(chunk))
    for t0 in range(0, L, step):
        t1 = min(L, t0 + step)
        xc = _f64(x[:, t0:t1])
        Bm, Cm, _, _ = project(xc, xc[None, :, :1], params["W_B"], params["W_C"], params.get("b_B"),
                               params.get("b_C"))
        xs = np.ascontiguousarray(xc[..., sel])
        delta, _ = discretize(xs, xs[None], w, bd)
        sig = expit(xs * w + bd) if delta_params else None
        gs = np.ascontiguousarray(_f64(gy[:, t0:t1])[..., sel])
        yc, G, st = core_param(As, xs, delta, gs, Bm, Cm, st, nthreads, drive, act, Dr, sig, scale)
        y[:, t0:t1] = yc
        for i in range(len(tot)):
            tot[i] += G[i]
    if st is None:
        st = tuple(np.zeros((B, Ds, N)) for _ in range(5 if delta_params else 3))
    if return_scale:
        return y, tuple(g.sum(0) for g in tot), st, tuple(s_.sum(0) for s_ in scale)
    return y, tuple(g.sum(0) for g in tot), st


# ------------------------------------------------------------------ linear attention

def la_scan_jvp(q, k, v, g, dq, dk, dv, dg, state=None, chunk=None, nthreads=None):
    """Decaying linear attention and its tangent flow (see pgf_oracle_la).
    q, k, g [B,H,L,dk]; v [B,H,L,dv]; dq, dk, dg [K,B,H,L,dk];
    dv [K,B,H,L,dv]; state = (S [B,H,dk,dv], dS [K,B,H,dk,dv]) or None.
    Returns (o [B,H,L,dv], do [K,B,H,L,dv], S_out, dS_out)."""
    lib = _load()
    B, H, L, DK = np.shape(q)
    DV = np.shape(v)[-1]
    K = np.shape(dq)[0]
    if state is None:
        S = np.zeros((B, H, DK, DV))
        dS = np.zeros((K, B, H, DK, DV))
    else:
        S = np.array(state[0], dtype=np.float64, copy=True, order="C")
        dS = np.array(state[1], dtype=np.float64, copy=True, order="C")
    assert S.shape == (B, H, DK, DV) and dS.shape == (K, B, H, DK, DV)
    o = np.empty((B, H, L, DV))
    do = np.empty((K, B, H, L, DV))
    step = max(1, L if not chunk else int(chunk))
    for t0 in range(0, L, step):
        t1 = min(L, t0 + step)
        a = [_f64(np.asarray(u)[..., t0:t1, :]) for u in (q, k, v, g, dq, dk, dv, dg)]
        oc = np.empty((B, H, t1 - t0, DV))
        doc = np.empty((K, B, H, t1 - t0, DV))
        rc = lib.pgf_oracle_la(B, H, t1 - t0, DK, DV, K, *[_dp(u) for u in a], _dp(S), _dp(dS), _dp(oc), _dp(doc),
                               _threads() if nthreads is None else nthreads)
        if rc != 0:
            raise RuntimeError("pgf_oracle_la failed")
        o[:, :, t0:t1] = oc
        do[:, :, :, t0:t1] = doc
    return o, do, S, dS
