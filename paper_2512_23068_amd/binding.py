"""Python binding of libpgf (argument marshalling only).

Every step of the scan runs in the HIP library ``libpgf.so`` built from
``csrc/``; this module checks tensor metadata, allocates outputs and the
workspace with torch, and passes raw device pointers and the current HIP
stream through the C ABI declared in ``include/pgf.h``.  There is no other
compute path: if the library is missing, every call raises.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpgf.so")

PGF_OK = 0
PGF_F32 = 0
PGF_BF16 = 1
DRIVES = {"euler": 0, "zoh": 1}
ACTIVATIONS = {"identity": 0, "silu": 1}
TIMING_KINDS = ("proj", "seg_aggregate", "carry", "scan_out", "state_io")

_c_f = ctypes.c_void_p


class PgfParams(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64), ("seqlen", ctypes.c_int64), ("d_inner", ctypes.c_int64),
        ("d_state", ctypes.c_int64), ("n_dirs", ctypes.c_int64),
        ("in_dtype", ctypes.c_int32), ("seg_len", ctypes.c_int32), ("chunk_segs", ctypes.c_int32),
        ("order", ctypes.c_int32),
        ("A", _c_f), ("w_delta", _c_f), ("b_delta", _c_f), ("W_B", _c_f), ("W_C", _c_f),
        ("b_B", _c_f), ("b_C", _c_f),
        ("h_in", _c_f), ("dh_in", _c_f), ("h_out", _c_f), ("dh_out", _c_f),
        ("workspace", _c_f), ("workspace_bytes", ctypes.c_size_t),
        ("d2h_in", _c_f), ("d2h_out", _c_f),
        ("drive", ctypes.c_int32), ("activation", ctypes.c_int32), ("D_res", _c_f), ("A_im", _c_f),
        ("n_groups", ctypes.c_int32), ("dt_rank", ctypes.c_int32), ("W_dx", _c_f), ("W_dt", _c_f),
        ("grad_D_res", _c_f), ("delta_flows", ctypes.c_int32), ("grad_w_delta", _c_f), ("grad_b_delta", _c_f),
    ]


class PgfLaParams(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64), ("heads", ctypes.c_int64), ("seqlen", ctypes.c_int64),
        ("d_key", ctypes.c_int64), ("d_value", ctypes.c_int64), ("n_dirs", ctypes.c_int64),
        ("seg_len", ctypes.c_int32), ("chunk_segs", ctypes.c_int32),
        ("S_in", _c_f), ("dS_in", _c_f), ("S_out", _c_f), ("dS_out", _c_f),
        ("workspace", _c_f), ("workspace_bytes", ctypes.c_size_t),
    ]


class PgfPlanInfo(ctypes.Structure):
    _fields_ = [
        ("n_per_thread", ctypes.c_int32), ("n_split", ctypes.c_int32), ("seg_len", ctypes.c_int32),
        ("chunk_segs", ctypes.c_int32), ("chunk_len", ctypes.c_int64), ("n_chunks", ctypes.c_int64),
        ("workspace_bytes", ctypes.c_size_t),
    ]


EXPORTED = ("pgf_workspace_bytes", "pgf_plan", "pgf_scan_jvp", "pgf_scan_jvp_noalloc", "pgf_scan_jvp2",
            "pgf_param_grads",
            "pgf_la_workspace_bytes", "pgf_la_plan", "pgf_la_scan_jvp", "pgf_status_string", "pgf_timing_enable",
            "pgf_timing_read")

_lib = None


def lib():
    """The loaded libpgf (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libpgf.so not found at {LIB_PATH}: build it with __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(PgfParams)
    L.pgf_workspace_bytes.restype = ctypes.c_size_t
    L.pgf_workspace_bytes.argtypes = [P]
    L.pgf_plan.restype = ctypes.c_int
    L.pgf_plan.argtypes = [P, ctypes.POINTER(PgfPlanInfo)]
    L.pgf_scan_jvp.restype = ctypes.c_int
    L.pgf_scan_jvp.argtypes = [ctypes.c_void_p, ctypes.c_void_p, P, ctypes.c_void_p, ctypes.c_void_p,
                               ctypes.c_void_p]
    L.pgf_scan_jvp_noalloc.restype = ctypes.c_int
    L.pgf_scan_jvp_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_void_p, P, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p]
    L.pgf_scan_jvp2.restype = ctypes.c_int
    L.pgf_scan_jvp2.argtypes = [ctypes.c_void_p, ctypes.c_void_p, P, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_void_p]
    L.pgf_param_grads.restype = ctypes.c_int
    L.pgf_param_grads.argtypes = [ctypes.c_void_p, ctypes.c_void_p, P, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    LP = ctypes.POINTER(PgfLaParams)
    L.pgf_la_workspace_bytes.restype = ctypes.c_size_t
    L.pgf_la_workspace_bytes.argtypes = [LP]
    L.pgf_la_plan.restype = ctypes.c_int
    L.pgf_la_plan.argtypes = [LP, ctypes.POINTER(PgfPlanInfo)]
    L.pgf_la_scan_jvp.restype = ctypes.c_int
    L.pgf_la_scan_jvp.argtypes = [ctypes.c_void_p] * 8 + [LP, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.pgf_status_string.restype = ctypes.c_char_p
    L.pgf_status_string.argtypes = [ctypes.c_int]
    L.pgf_timing_enable.restype = ctypes.c_int
    L.pgf_timing_enable.argtypes = [ctypes.c_int]
    L.pgf_timing_read.restype = ctypes.c_int
    L.pgf_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    _lib = L
    return L


def status_string(code: int) -> str:
    return lib().pgf_status_string(int(code)).decode()


def _check(code: int):
    if code != PGF_OK:
        raise RuntimeError(status_string(code))


def make_params(B, L, D, N, K, in_dtype="f32", seg_len=0, chunk_segs=0, order=1, drive="euler",
                act="identity", delta_flows=False) -> PgfParams:
    p = PgfParams()
    p.batch, p.seqlen, p.d_inner, p.d_state, p.n_dirs = int(B), int(L), int(D), int(N), int(K)
    p.in_dtype = PGF_BF16 if in_dtype in ("bf16", torch.bfloat16) else PGF_F32
    p.seg_len, p.chunk_segs, p.order = int(seg_len), int(chunk_segs), int(order)
    p.drive, p.activation = DRIVES[drive], ACTIVATIONS[act]
    p.delta_flows = 1 if delta_flows else 0
    return p


def workspace_bytes(B, L, D, N, K, in_dtype="f32", seg_len=0, chunk_segs=0, order=1, drive="euler",
                    act="identity", delta_flows=False) -> int:
    return int(lib().pgf_workspace_bytes(ctypes.byref(make_params(B, L, D, N, K, in_dtype, seg_len, chunk_segs,
                                                                  order, drive, act, delta_flows))))


def plan(B, L, D, N, K, in_dtype="f32", seg_len=0, chunk_segs=0, order=1, drive="euler", act="identity",
         complex_a=False, groups=1, dt_rank=0, delta_flows=False) -> dict:
    """The tiling a call would use (complex_a: with a complex transition;
    the planner only tests A_im for NULL, the pointer is never read;
    delta_flows: the parameter flows of the step size's parameters)."""
    info = PgfPlanInfo()
    pr = make_params(B, L, D, N, K, in_dtype, seg_len, chunk_segs, order, drive, act, delta_flows)
    pr.n_groups = int(groups)
    pr.dt_rank = int(dt_rank)
    if complex_a:
        pr.A_im = 1
    _check(lib().pgf_plan(ctypes.byref(pr), ctypes.byref(info)))
    return {f: getattr(info, f) for f, _ in PgfPlanInfo._fields_}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev_param(v, shape, device, name):
    if v is None:
        return None
    if not isinstance(v, torch.Tensor):
        v = torch.as_tensor(v)
    if tuple(v.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(v.shape)}")
    return v.to(device=device, dtype=torch.float32).contiguous()


def _model_params(pr, params, D, dev, keep):
    """Moves the model parameters to the device as f32 and stores their
    pointers in pr; returns N."""
    A = _dev_param(params["A"], (D, params["A"].shape[1]), dev, "A")
    N = A.shape[1]
    G = int(params.get("n_groups") or 1)
    pr.n_groups = G
    # Low-rank step size: W_dx [D,R] and W_dt [R,D] replace w_delta.
    R = 0 if params.get("W_dt") is None else int(params["W_dt"].shape[0])
    pr.dt_rank = R
    vals = {"A": A}
    for name, shape in (("w_delta", (D,)), ("b_delta", (D,)), ("W_B", (D, G * N)), ("W_C", (D, G * N)),
                        ("b_B", (G * N,)), ("b_C", (G * N,)), ("W_dx", (D, R)), ("W_dt", (R, D))):
        if R and name == "w_delta":
            continue
        vals[name] = _dev_param(params.get(name), shape, dev, name)
    for name, v in vals.items():
        keep.append(v)
        setattr(pr, name, None if v is None else v.data_ptr())
    return N


def _dev_state_c(v, shape, device, name):
    """A complex state (complex64 on the device, interleaved real/imag)."""
    if v is None:
        return None
    if not isinstance(v, torch.Tensor):
        v = torch.as_tensor(v)
    if tuple(v.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(v.shape)}")
    return v.to(device=device, dtype=torch.complex64).contiguous()


def _checked_workspace(workspace, nbytes, dev):
    """The caller's workspace (a contiguous uint8 tensor on dev of at least
    nbytes) or, when None, a new one."""
    if workspace is None:
        return torch.empty(max(nbytes, 1), device=dev, dtype=torch.uint8)
    if not (isinstance(workspace, torch.Tensor) and workspace.dtype == torch.uint8 and workspace.device == dev
            and workspace.is_contiguous()):
        raise ValueError(f"workspace: expected a contiguous uint8 tensor on {dev}")
    if workspace.numel() < nbytes:
        raise ValueError(f"workspace: {workspace.numel()} bytes, the call needs {nbytes}")
    return workspace


def _workspace(L_, pr, workspace, dev):
    nbytes = int(L_.pgf_workspace_bytes(ctypes.byref(pr)))
    if nbytes == 0:
        _check(L_.pgf_plan(ctypes.byref(pr), ctypes.byref(PgfPlanInfo())))
    workspace = _checked_workspace(workspace, nbytes, dev)
    pr.workspace, pr.workspace_bytes = workspace.data_ptr(), workspace.numel()
    return workspace


def _check_out(t, shape, dev, name):
    """A caller-provided output must be exactly what the kernels write: the
    library only sees its address."""
    if not (isinstance(t, torch.Tensor) and t.dtype == torch.float32 and t.device == dev
            and tuple(t.shape) == tuple(shape) and t.is_contiguous()):
        got = (tuple(t.shape), t.dtype, str(t.device), t.is_contiguous()) if isinstance(t, torch.Tensor) else type(t)
        raise ValueError(f"{name}: expected a contiguous float32 tensor of shape {tuple(shape)} on {dev}, got {got}")
    return t


def _outputs(out, shapes, names, dev):
    """Checked caller outputs, or new ones."""
    if out is None:
        return tuple(torch.empty(s, device=dev, dtype=torch.float32) for s in shapes)
    if isinstance(out, torch.Tensor):
        out = (out,)
    out = tuple(out)
    if len(out) != len(shapes):
        raise ValueError(f"out: expected {len(shapes)} tensors ({', '.join(names)}), got {len(out)}")
    return tuple(_check_out(t, s, dev, n) for t, s, n in zip(out, shapes, names))


def _on_stream(stream, dev):
    """Context in which the call allocates its temporaries and launches:
    the caller's torch.cuda.Stream when given (so that the caching allocator
    ties every temporary to the stream the kernels run on), else the current
    stream of dev."""
    if stream is None:
        return contextlib.nullcontext()
    if not isinstance(stream, torch.cuda.Stream):
        raise ValueError("stream: expected a torch.cuda.Stream (or None for the current stream)")
    if stream.device != dev:
        raise ValueError(f"stream: on {stream.device}, the tensors are on {dev}")
    return torch.cuda.stream(stream)


def _scan(x, dx, params, order, h_in, dh_in, d2h_in, return_state, seg_len, chunk_segs, workspace, out, stream,
          drive="euler", act="identity"):
    if not (isinstance(x, torch.Tensor) and isinstance(dx, torch.Tensor) and x.is_cuda and dx.is_cuda):
        raise ValueError("x and dx must be device tensors")
    if dx.device != x.device:
        raise ValueError("x and dx must be on the same device")
    with torch.cuda.device(x.device), _on_stream(stream, x.device):
        return _scan_on(x, dx, params, order, h_in, dh_in, d2h_in, return_state, seg_len, chunk_segs, workspace,
                        out, drive, act)


def _scan_on(x, dx, params, order, h_in, dh_in, d2h_in, return_state, seg_len, chunk_segs, workspace, out, drive,
             act):
    L_ = lib()
    if x.dtype not in (torch.float32, torch.bfloat16) or dx.dtype != x.dtype:
        raise ValueError("x and dx must both be float32 or both bfloat16")
    if x.dim() != 3 or dx.dim() != 4 or tuple(dx.shape[1:]) != tuple(x.shape):
        raise ValueError(f"shapes: x [B,L,D], dx [K,B,L,D]; got {tuple(x.shape)}, {tuple(dx.shape)}")
    x = x.contiguous()
    dx = dx.contiguous()
    B, L, D = x.shape
    K = dx.shape[0]
    if order == 2 and K != 2:
        raise ValueError("the second-order scan takes exactly two directions (dx of shape [2,B,L,D])")
    dev = x.device
    pr = make_params(B, L, D, params["A"].shape[1], K, "bf16" if x.dtype == torch.bfloat16 else "f32", seg_len,
                     chunk_segs, order, drive, act)
    keep = []
    N = _model_params(pr, params, D, dev, keep)
    D_res = _dev_param(params.get("D_res"), (D,), dev, "D_res")
    keep.append(D_res)
    pr.D_res = None if D_res is None else D_res.data_ptr()
    A_im = _dev_param(params.get("A_im"), (D, N), dev, "A_im")
    keep.append(A_im)
    pr.A_im = None if A_im is None else A_im.data_ptr()
    cplx = A_im is not None
    if cplx:
        h_in = _dev_state_c(h_in, (B, D, N), dev, "h_in")
        dh_in = _dev_state_c(dh_in, (K, B, D, N), dev, "dh_in")
    else:
        h_in = _dev_param(h_in, (B, D, N), dev, "h_in")
        dh_in = _dev_param(dh_in, (K, B, D, N), dev, "dh_in")
    d2h_in = _dev_param(d2h_in, (B, D, N), dev, "d2h_in")
    pr.h_in = None if h_in is None else h_in.data_ptr()
    pr.dh_in = None if dh_in is None else dh_in.data_ptr()
    pr.d2h_in = None if d2h_in is None else d2h_in.data_ptr()
    states = ()
    if return_state:
        sdt = torch.complex64 if cplx else torch.float32
        h_out = torch.empty((B, D, N), device=dev, dtype=sdt)
        dh_out = torch.empty((K, B, D, N), device=dev, dtype=sdt)
        pr.h_out, pr.dh_out = h_out.data_ptr(), dh_out.data_ptr()
        states = (h_out, dh_out)
        if order == 2:
            d2h_out = torch.empty((B, D, N), device=dev, dtype=torch.float32)
            pr.d2h_out = d2h_out.data_ptr()
            states = states + (d2h_out,)
    if order == 2:
        outs = _outputs(out, ((B, L, D), (K, B, L, D), (B, L, D)), ("y", "dy", "d2y"), dev)
    else:
        outs = _outputs(out, ((B, L, D), (K, B, L, D)), ("y", "dy"), dev)
    workspace = _workspace(L_, pr, workspace, dev)
    st = torch.cuda.current_stream(dev).cuda_stream
    if order == 2:
        rc = L_.pgf_scan_jvp2(_ptr(x), _ptr(dx), ctypes.byref(pr), _ptr(outs[0]), _ptr(outs[1]), _ptr(outs[2]),
                              ctypes.c_void_p(st))
    else:
        rc = L_.pgf_scan_jvp(_ptr(x), _ptr(dx), ctypes.byref(pr), _ptr(outs[0]), _ptr(outs[1]),
                             ctypes.c_void_p(st))
    _check(rc)
    return outs + states


def scan_jvp(x: torch.Tensor, dx: torch.Tensor, params: dict, *, h_in=None, dh_in=None, return_state=False,
             seg_len=0, chunk_segs=0, workspace=None, out=None, stream=None, drive="euler", act="identity"):
    """Fused primal + tangent scan on the GPU.

    x [B,L,D] and dx [K,B,L,D]: float32 or bfloat16 CUDA tensors (same dtype).
    params: A, W_B, W_C [D,N]; w_delta, b_delta [D]; optional b_B, b_C [N],
    D_res [D] (residual weight of the output map), A_im [D,N] (imaginary
    part of a complex transition; the states are then complex64),
    n_groups (W_B, W_C [D,G*N], b_B, b_C [G*N]) and W_dx [D,R], W_dt [R,D]
    (low-rank step size; w_delta is then not used).
    drive: "euler" or "zoh"; act: "identity" or "silu" (the variants need
    N <= 16 and K <= 2).
    Returns (y [B,L,D], dy [K,B,L,D]) in float32, plus (h_out [B,D,N],
    dh_out [K,B,D,N]) when return_state.  Asynchronous on the current stream.
    """
    return _scan(x, dx, params, 1, h_in, dh_in, None, return_state, seg_len, chunk_segs, workspace, out, stream,
                 drive, act)


def scan_jvp_noalloc(x: torch.Tensor, dx: torch.Tensor, params: dict, out, *, h_in=None, dh_in=None, seg_len=0,
                     chunk_segs=0, stream=None, drive="euler", act="identity"):
    """scan_jvp through pgf_scan_jvp_noalloc: the library takes its workspace
    from a static per-GPU array (PGF_SCRATCH_BYTES) instead of the caller.

    out = (y [B,L,D], dy [K,B,L,D]) float32 on the device, required; with
    parameters and states already contiguous float32 on the device the
    binding allocates nothing either.  Returns out.  Calls that overlap on
    one GPU race (they share the array)."""
    if not (isinstance(x, torch.Tensor) and isinstance(dx, torch.Tensor) and x.is_cuda and dx.is_cuda):
        raise ValueError("x and dx must be device tensors")
    if out is None:
        raise ValueError("out: the caller provides y and dy")
    with torch.cuda.device(x.device), _on_stream(stream, x.device):
        L_ = lib()
        if x.dtype not in (torch.float32, torch.bfloat16) or dx.dtype != x.dtype:
            raise ValueError("x and dx must both be float32 or both bfloat16")
        if x.dim() != 3 or dx.dim() != 4 or tuple(dx.shape[1:]) != tuple(x.shape) or dx.device != x.device:
            raise ValueError(f"shapes: x [B,L,D], dx [K,B,L,D]; got {tuple(x.shape)}, {tuple(dx.shape)}")
        if not (x.is_contiguous() and dx.is_contiguous()):
            raise ValueError("x and dx must be contiguous")
        B, L, D = x.shape
        K = dx.shape[0]
        dev = x.device
        pr = make_params(B, L, D, params["A"].shape[1], K, "bf16" if x.dtype == torch.bfloat16 else "f32", seg_len,
                         chunk_segs, 1, drive, act)
        keep = []
        N = _model_params(pr, params, D, dev, keep)
        D_res = _dev_param(params.get("D_res"), (D,), dev, "D_res")
        keep.append(D_res)
        pr.D_res = None if D_res is None else D_res.data_ptr()
        if params.get("A_im") is not None:
            raise ValueError("scan_jvp_noalloc: real transitions only")
        h_in = _dev_param(h_in, (B, D, N), dev, "h_in")
        dh_in = _dev_param(dh_in, (K, B, D, N), dev, "dh_in")
        pr.h_in = None if h_in is None else h_in.data_ptr()
        pr.dh_in = None if dh_in is None else dh_in.data_ptr()
        y, dy = _outputs(out, ((B, L, D), (K, B, L, D)), ("y", "dy"), dev)
        st = torch.cuda.current_stream(dev).cuda_stream
        _check(L_.pgf_scan_jvp_noalloc(_ptr(x), _ptr(dx), ctypes.byref(pr), _ptr(y), _ptr(dy), ctypes.c_void_p(st)))
        return y, dy


def scan_jvp2(x: torch.Tensor, dx: torch.Tensor, params: dict, *, h_in=None, dh_in=None, d2h_in=None,
              return_state=False, seg_len=0, chunk_segs=0, workspace=None, out=None, stream=None):
    """Second-order flow on the GPU along v = dx[0], w = dx[1] (dx [2,B,L,D]).

    Returns (y [B,L,D], dy [2,B,L,D], d2y [B,L,D]) in float32: the primal,
    both first-order directional derivatives and the mixed second
    directional derivative; plus (h_out, dh_out, d2h_out) when return_state.
    """
    return _scan(x, dx, params, 2, h_in, dh_in, d2h_in, return_state, seg_len, chunk_segs, workspace, out,
                 stream)


def param_grads(x: torch.Tensor, gy: torch.Tensor, params: dict, *, h_in=None, gamma_in=None, grads=None,
                return_state=False, seg_len=0, chunk_segs=0, workspace=None, out=None, stream=None,
                drive="euler", act="identity", delta_params=False):
    """Primal scan with the parameter-sensitivity flows and online gradient
    accumulation against the adjoint signal gy = dl/dy, on the GPU.

    x [B,L,D] float32 or bfloat16 and gy [B,L,D] float32, CUDA tensors.
    grads: optional (grad_A, grad_B, grad_C), each [D,N] float32 on the
    device, which are ADDED to in place (zeros are allocated when None).
    gamma_in: optional [2,B,D,N] entry state of the flows (dh/dA, dh/dB;
    [4,B,D,N] with dh/dw_delta and dh/db_delta when delta_params).
    Returns (y [B,L,D], grad_A, grad_B, grad_C), plus (h_out [B,D,N],
    gamma_out [2,B,D,N]) when return_state.  grad_B and grad_C are the
    gradients of per-lane offsets of B and C; their sums over d are
    dl/db_B and dl/db_C.  drive: "euler" or "zoh" (the zero-order-hold drive,
    whose derivative in A enters dl/dA).  act ("identity" or "silu") and
    params["D_res"] (optional [D]) set the output map y = act(C h + D_res x);
    with D_res the gradients gain a fourth, grad_D_res [D] (grads then holds
    four tensors when given).  delta_params adds the flows of the step
    size's parameters: the gradients then end with grad_w_delta and
    grad_b_delta [D].  Asynchronous on the current stream.
    """
    if not (isinstance(x, torch.Tensor) and isinstance(gy, torch.Tensor) and x.is_cuda and gy.is_cuda):
        raise ValueError("x and gy must be device tensors")
    if gy.device != x.device:
        raise ValueError("x and gy must be on the same device")
    with torch.cuda.device(x.device), _on_stream(stream, x.device):
        return _param_grads_on(x, gy, params, h_in, gamma_in, grads, return_state, seg_len, chunk_segs, workspace,
                               out, drive, act, delta_params)


def _param_grads_on(x, gy, params, h_in, gamma_in, grads, return_state, seg_len, chunk_segs, workspace, out,
                    drive, act, delta_params):
    L_ = lib()
    if x.dtype not in (torch.float32, torch.bfloat16) or gy.dtype != torch.float32:
        raise ValueError("x must be float32 or bfloat16 and gy float32")
    if x.dim() != 3 or tuple(gy.shape) != tuple(x.shape):
        raise ValueError(f"shapes: x and gy [B,L,D]; got {tuple(x.shape)}, {tuple(gy.shape)}")
    x = x.contiguous()
    gy = gy.contiguous()
    B, L, D = x.shape
    dev = x.device
    pr = make_params(B, L, D, params["A"].shape[1], 2, "bf16" if x.dtype == torch.bfloat16 else "f32", seg_len,
                     chunk_segs, 3, drive, act, delta_params)
    keep = []
    N = _model_params(pr, params, D, dev, keep)
    if params.get("A_im") is not None:
        raise ValueError("param_grads: real transitions only")
    D_res = _dev_param(params.get("D_res"), (D,), dev, "D_res")
    keep.append(D_res)
    pr.D_res = None if D_res is None else D_res.data_ptr()
    shapes = [(D, N)] * 3 + ([(D,)] if D_res is not None else []) + ([(D,), (D,)] if delta_params else [])
    ng = 4 if delta_params else 2     # planes of gamma_in / gamma_out
    h_in = _dev_param(h_in, (B, D, N), dev, "h_in")
    gamma_in = _dev_param(gamma_in, (ng, B, D, N), dev, "gamma_in")
    pr.h_in = None if h_in is None else h_in.data_ptr()
    pr.dh_in = None if gamma_in is None else gamma_in.data_ptr()
    states = ()
    if return_state:
        h_out = torch.empty((B, D, N), device=dev, dtype=torch.float32)
        g_out = torch.empty((ng, B, D, N), device=dev, dtype=torch.float32)
        pr.h_out, pr.dh_out = h_out.data_ptr(), g_out.data_ptr()
        states = (h_out, g_out)
    if grads is None:
        grads = tuple(torch.zeros(sh, device=dev, dtype=torch.float32) for sh in shapes)
    else:
        grads = tuple(grads)
        if len(grads) != len(shapes) or not all(
                isinstance(g, torch.Tensor) and g.dtype == torch.float32 and g.device == dev
                and tuple(g.shape) == sh and g.is_contiguous() for g, sh in zip(grads, shapes)):
            raise ValueError(f"grads: {len(shapes)} contiguous float32 tensors of shapes {shapes} on {dev}")
    if D_res is not None:
        pr.grad_D_res = grads[3].data_ptr()
    if delta_params:
        pr.grad_w_delta, pr.grad_b_delta = grads[-2].data_ptr(), grads[-1].data_ptr()
    y, = _outputs(out, ((B, L, D),), ("y",), dev)
    workspace = _workspace(L_, pr, workspace, dev)
    st = torch.cuda.current_stream(dev).cuda_stream
    rc = L_.pgf_param_grads(_ptr(x), _ptr(gy), ctypes.byref(pr), _ptr(y), _ptr(grads[0]), _ptr(grads[1]),
                            _ptr(grads[2]), ctypes.c_void_p(st))
    _check(rc)
    return (y,) + grads + states


def make_la_params(B, H, L, DK, DV, K, seg_len=0, chunk_segs=0) -> PgfLaParams:
    p = PgfLaParams()
    p.batch, p.heads, p.seqlen, p.d_key, p.d_value, p.n_dirs = int(B), int(H), int(L), int(DK), int(DV), int(K)
    p.seg_len, p.chunk_segs = int(seg_len), int(chunk_segs)
    return p


def la_plan(B, H, L, DK, DV, K, seg_len=0, chunk_segs=0) -> dict:
    info = PgfPlanInfo()
    _check(lib().pgf_la_plan(ctypes.byref(make_la_params(B, H, L, DK, DV, K, seg_len, chunk_segs)),
                             ctypes.byref(info)))
    return {f: getattr(info, f) for f, _ in PgfPlanInfo._fields_}


def la_scan_jvp(q, k, v, g, dq, dk, dv, dg, *, S_in=None, dS_in=None, return_state=False, seg_len=0,
                chunk_segs=0, workspace=None, out=None, stream=None):
    """Decaying linear attention and its tangent flow on the GPU.

    q, k, g [B,H,L,dk]; v [B,H,L,dv]; dq, dk, dg [K,B,H,L,dk]; dv [K,B,H,L,dv]:
    float32 CUDA tensors (g is the log-decay).  Returns (o [B,H,L,dv],
    do [K,B,H,L,dv]), plus (S_out [B,H,dk,dv], dS_out [K,B,H,dk,dv]) when
    return_state.  Asynchronous on the current stream.
    """
    ts = [q, k, v, g, dq, dk, dv, dg]
    if not all(isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.float32 for t in ts):
        raise ValueError("q, k, v, g, dq, dk, dv, dg must be float32 device tensors")
    if any(t.device != q.device for t in ts):
        raise ValueError("q, k, v, g, dq, dk, dv, dg must be on one device")
    with torch.cuda.device(q.device), _on_stream(stream, q.device):
        return _la_scan_jvp_on(ts, S_in, dS_in, return_state, seg_len, chunk_segs, workspace, out)


def _la_scan_jvp_on(ts, S_in, dS_in, return_state, seg_len, chunk_segs, workspace, out):
    L_ = lib()
    q, k, v, g, dq, dk, dv, dg = ts
    if q.dim() != 4 or dq.dim() != 5:
        raise ValueError("shapes: q, k, g [B,H,L,dk], v [B,H,L,dv], tangents with a leading K")
    B, H, L, DK = q.shape
    DV = v.shape[-1]
    K = dq.shape[0]
    for t, shape in ((k, (B, H, L, DK)), (g, (B, H, L, DK)), (v, (B, H, L, DV)), (dq, (K, B, H, L, DK)),
                     (dk, (K, B, H, L, DK)), (dg, (K, B, H, L, DK)), (dv, (K, B, H, L, DV))):
        if tuple(t.shape) != shape:
            raise ValueError(f"expected shape {shape}, got {tuple(t.shape)}")
    ts = [t.contiguous() for t in ts]
    dev = q.device
    pr = make_la_params(B, H, L, DK, DV, K, seg_len, chunk_segs)
    S_in = _dev_param(S_in, (B, H, DK, DV), dev, "S_in")
    dS_in = _dev_param(dS_in, (K, B, H, DK, DV), dev, "dS_in")
    pr.S_in = None if S_in is None else S_in.data_ptr()
    pr.dS_in = None if dS_in is None else dS_in.data_ptr()
    states = ()
    if return_state:
        S_out = torch.empty((B, H, DK, DV), device=dev, dtype=torch.float32)
        dS_out = torch.empty((K, B, H, DK, DV), device=dev, dtype=torch.float32)
        pr.S_out, pr.dS_out = S_out.data_ptr(), dS_out.data_ptr()
        states = (S_out, dS_out)
    nbytes = int(L_.pgf_la_workspace_bytes(ctypes.byref(pr)))
    if nbytes == 0:
        _check(L_.pgf_la_plan(ctypes.byref(pr), ctypes.byref(PgfPlanInfo())))
    o, do = _outputs(out, ((B, H, L, DV), (K, B, H, L, DV)), ("o", "do"), dev)
    workspace = _checked_workspace(workspace, nbytes, dev)
    pr.workspace, pr.workspace_bytes = workspace.data_ptr(), workspace.numel()
    st = torch.cuda.current_stream(dev).cuda_stream
    rc = L_.pgf_la_scan_jvp(*[_ptr(t) for t in ts], ctypes.byref(pr), _ptr(o), _ptr(do), ctypes.c_void_p(st))
    _check(rc)
    return (o, do) + states


def timing_enable(on: bool = True):
    _check(lib().pgf_timing_enable(1 if on else 0))


def timing_read() -> dict:
    ms = (ctypes.c_double * len(TIMING_KINDS))()
    n = (ctypes.c_int64 * len(TIMING_KINDS))()
    _check(lib().pgf_timing_read(ms, n))
    return {k: (ms[i], n[i]) for i, k in enumerate(TIMING_KINDS)}
