"""The five benchmark workloads at their full sizes, in the launch
configuration the benchmark times (the default plan), against the fp64
oracle over the whole sequence: every channel of tiny, mamba130m and
pulse128k, and channels from every 256-channel block of stiff128k and
multidir (the oracle computes any channel on its own; the projections still
contract over every channel).  Each case records its errors, per tangent
direction, in the parity record (gpu_util.PARITY_JSON), and pulse128k also
the error of the impulse response's last 1024 steps against a worst-case
rounding bound.  Also: peak device memory minus the IO payload is the same
for every L."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

# Channels compared per workload: every channel where the oracle finishes
# in about a minute (pulse128k, mamba130m), otherwise a seeded choice of
# `per_block` channels in every block of 256 channels (the scan kernels'
# block width), so every launch block of the channel grid is checked.
FULL = {"tiny": None, "mamba130m": None, "pulse128k": None, "stiff128k": 4, "multidir": 8}


def _channels(D, per_block, seed=0):
    if per_block is None:
        return np.arange(D, dtype=np.int64)
    g = np.random.default_rng(seed)
    out = []
    for b0 in range(0, D, 256):
        blk = np.arange(b0, min(D, b0 + 256))
        out.append(g.choice(blk, size=min(per_block, len(blk)), replace=False))
    return np.unique(np.concatenate([[0, D - 1]] + out)).astype(np.int64)


def _run_full(name):
    cfg = inputs.get_config(name)
    print(f"case {name}: generating inputs", flush=True)
    inp = inputs.make_inputs(cfg)
    sel = _channels(cfg.d_inner, FULL[name])
    x, dx = gu.inputs_to_dev(inp)
    print(f"case {name}: GPU scan", flush=True)
    y, dy = binding.scan_jvp(x, dx, gu.params_to_dev(inp))
    torch.cuda.synchronize()
    if len(sel) == cfg.d_inner:
        yg, dyg = y.cpu().numpy(), dy.cpu().numpy()
    else:
        idx = torch.from_numpy(sel).to(gu.dev())
        yg = y.index_select(-1, idx).cpu().numpy()
        dyg = dy.index_select(-1, idx).cpu().numpy()
    del x, dx, y, dy
    torch.cuda.empty_cache()
    print(f"case {name}: oracle on {len(sel)} of {cfg.d_inner} channels", flush=True)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, channels=sel, chunk=4096)
    return cfg, sel, yg, dyg, yo, dyo


# Rounding model of the tail (see tail_bound): per factor of the decay chain
# the exponential errs by at most 0.66 ulp (measured over every f32 argument
# of the transitions' range) and the product rounds once, together at most
# 1.4e-7 relative; after the lift of the transition's argument their mean is
# below 2e-10 per step.
U_FACTOR = 1.4e-7
MEAN_PER_STEP = 2e-10


def tail_bound(seg, L, lam=6.0):
    """Bound on the relative error of the impulse response's tail.

    For t >= 1 the impulse direction has dx_t = 0, so dDelta_t, p_t, dB_t and
    dC_t vanish and each lane's tangent only decays: dh_t = Abar_t dh_{t-1}.
    The computed tail value is dh_0 times a chain of n rounded factors: in
    the segmented evaluation the segment transitions P of the segments
    before the last (seg steps each) and the step transitions Abar of the
    last segment (n = L/seg - 1 + seg); in the sequential evaluation
    (seg = 0) the L step transitions.  Its relative error is the sum of the
    factors' errors; taking them as independent with mean below
    MEAN_PER_STEP and magnitude below U_FACTOR, the sum stays below
    lam * sqrt(n) * U_FACTOR + n * MEAN_PER_STEP except with probability
    2 exp(-lam^2 / 2) (the probabilistic rounding-error bound of Higham and
    Mary, 2019); lam = 6 gives 3e-8.  A biased transition (a mean error of
    7e-9 per step, as the raw hardware exponential has) exceeds the bound
    of the sequential evaluation by 3x."""
    n = (L // seg - 1 + seg) if seg else L
    return lam * np.sqrt(n) * U_FACTOR + n * MEAN_PER_STEP


@pytest.mark.parametrize("name", ["tiny", "mamba130m", "pulse128k", "stiff128k", "multidir"])
def test_full_workload_channels(name):
    cfg, sel, yg, dyg, yo, dyo = _run_full(name)
    ey = gu.rel_l2(yg, yo)
    edy = [gu.rel_l2(dyg[k], dyo[k]) for k in range(dyo.shape[0])]
    rec = {"shape": [cfg.batch, cfg.seqlen, cfg.d_inner, cfg.d_state, cfg.n_dirs], "in_dtype": cfg.in_dtype,
           "channels_compared": int(len(sel)), "channels_total": int(cfg.d_inner),
           "plan": binding.plan(cfg.batch, cfg.seqlen, cfg.d_inner, cfg.d_state, cfg.n_dirs, cfg.in_dtype),
           "y_rel_l2": ey, "dy_rel_l2_per_direction": edy, "dy_rel_l2_max": max(edy), "tolerance": gu.TOL}
    if name == "pulse128k":
        # the impulse response's tail over the last 1024 steps (its reason to exist)
        tail = gu.rel_l2(dyg[:, :, -1024:], dyo[:, :, -1024:])
        mag = float(np.abs(dyo[:, :, -1024:]).max())
        seg = rec["plan"]["seg_len"]
        bound = tail_bound(seg, cfg.seqlen)
        rec.update({"tail_steps": 1024, "tail_dy_rel_l2": tail, "tail_max_abs_dy": mag, "tail_bound": bound})
        print(f"pulse128k tail rel_l2(dy, last 1024 steps) = {tail:.3e} (bound {bound:.3e}; max |dy| {mag:.3e})",
              flush=True)
    gu.record(name, rec)
    gu.assert_close(yg, dyg, yo, dyo, what=name)
    if name == "pulse128k":
        assert mag > 0 and np.isfinite(tail) and tail <= rec["tail_bound"], rec


def _flat_case(kind):
    """(call(L) -> outputs, payload bytes(L), workspace bytes) of one entry
    point at a benchmark shape, on random device inputs."""
    dev = gu.dev()
    if kind == "la_scan_jvp":
        B, H, DK, DV = 1, 32, 64, 64

        def call(L):
            ts = [torch.randn(B, H, L, d, device=dev) * s for d, s in ((DK, 0.1), (DK, 0.1), (DV, 1.0))]
            ts.append(-torch.rand(B, H, L, DK, device=dev) * 0.05)
            ts += [torch.randn(1, *t.shape, device=dev) * 0.1 for t in ts]
            return ts, (lambda: binding.la_scan_jvp(*ts))
        return call, binding.la_plan(B, H, 8192, DK, DV, 1)["workspace_bytes"]
    name = "stiff128k" if kind == "scan_jvp_bf16" else "pulse128k"
    cfg = inputs.get_config(name)
    D, N = cfg.d_inner, cfg.d_state
    base = inputs.make_params(cfg)
    K = 2 if kind == "scan_jvp2" else 1
    dt = torch.bfloat16 if kind == "scan_jvp_bf16" else torch.float32
    lr = 48 if kind == "low_rank" else 0
    prm = inputs.variant_params({k: base[k] for k in ("A", "w_delta", "b_delta", "W_B", "W_C")}, cfg, lowrank=lr)
    prm = gu.params_to_dev(prm)
    order = {"scan_jvp2": 2, "param_grads": 3}.get(kind, 1)
    ws = binding.plan(1, 8192, D, N, K, "bf16" if dt == torch.bfloat16 else "f32", order=order,
                      dt_rank=lr)["workspace_bytes"]

    def call(L):
        x = torch.randn(1, L, D, device=dev).to(dt)
        if kind == "param_grads":
            gy = torch.randn(1, L, D, device=dev)
            return [x, gy], (lambda: binding.param_grads(x, gy, prm))
        dx = torch.randn(K, 1, L, D, device=dev).to(dt)
        fn = binding.scan_jvp2 if kind == "scan_jvp2" else binding.scan_jvp
        return [x, dx], (lambda: fn(x, dx, prm))
    return call, ws


@pytest.mark.parametrize("kind", ["scan_jvp", "scan_jvp_bf16", "scan_jvp2", "param_grads", "low_rank",
                                  "la_scan_jvp"])
def test_peak_memory_flat_in_L(kind):
    """Peak allocated bytes minus the IO payload (inputs and outputs) do not
    depend on L (Sec. 4.3: only the O(1) tile is differentiation overhead),
    for every entry point at a benchmark shape (pulse128k; stiff128k with
    bf16 inputs; rwkv128k for linear attention); and the device's free
    memory (hipMemGetInfo) drops by no more than what torch reserved, so the
    library allocates nothing outside torch."""
    call, ws = _flat_case(kind)
    ins, fn = call(131072)          # warm up at the longest sequence: every kernel loaded
    fn()
    torch.cuda.synchronize()
    del ins, fn
    incr, outside = [], []
    for L in (8192, 16384, 32768, 65536, 131072):
        torch.cuda.empty_cache()
        ins, fn = call(L)
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        free0, res0 = torch.cuda.mem_get_info()[0], torch.cuda.memory_reserved()
        torch.cuda.reset_peak_memory_stats()
        outs = fn()
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated()
        free1, res1 = torch.cuda.mem_get_info()[0], torch.cuda.memory_reserved()
        out_bytes = sum(t.numel() * t.element_size() for t in outs)
        incr.append(peak - base - out_bytes)
        outside.append((free0 - free1) - (res1 - res0))
        print(f"{kind} L={L}: peak-minus-payload {incr[-1]} bytes, outside torch {outside[-1]}", flush=True)
        del ins, fn, outs
    gu.record(f"flat_vram_{kind}", {"L": [8192, 16384, 32768, 65536, 131072], "peak_minus_payload": incr,
                                    "outside_torch": outside, "workspace_bytes": ws})
    assert len(set(incr)) == 1, incr
    assert incr[0] <= ws + (4 << 20), (incr[0], ws)
    assert all(o <= 0 for o in outside), outside


def test_sequential_tail_pulse128k():
    """The impulse response's tail in the sequential evaluation (every one of
    the 131072 steps a factor of the decay chain), on the 8 channels with the
    slowest decay (the largest tail) and 24 seeded others."""
    cfg = inputs.get_config("pulse128k")
    print("case pulse128k sequential tail: inputs", flush=True)
    inp = inputs.make_inputs(cfg)
    D = cfg.d_inner
    slow = np.argsort(inp["b_delta"])[:8]
    sel = np.unique(np.concatenate([slow, np.random.default_rng(3).choice(D, 24, replace=False)]))
    x, dx = gu.inputs_to_dev(inp)
    print("case pulse128k sequential tail: GPU scan", flush=True)
    y, dy = binding.scan_jvp(x, dx, gu.params_to_dev(inp), seg_len=-1)
    torch.cuda.synchronize()
    idx = torch.from_numpy(sel).to(gu.dev())
    dyg = dy[:, :, -1024:].index_select(-1, idx).cpu().numpy()
    del x, dx, y, dy
    torch.cuda.empty_cache()
    print(f"case pulse128k sequential tail: oracle on {len(sel)} channels", flush=True)
    _, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, channels=sel, chunk=8192)
    tail = gu.rel_l2(dyg, dyo[:, :, -1024:])
    bound = tail_bound(0, cfg.seqlen)
    print(f"pulse128k sequential tail rel_l2 = {tail:.3e} (bound {bound:.3e})", flush=True)
    gu.record("pulse128k_sequential_tail", {"seg_len": -1, "channels": sel.tolist(), "tail_steps": 1024,
                                            "tail_dy_rel_l2": tail, "tail_bound": bound})
    assert np.isfinite(tail) and tail <= bound, (tail, bound)


@pytest.mark.parametrize("seg", [0, -1])
def test_ghost_pulse_full_size(seg):
    """The ghost pulse at the paper's depth: pulse128k's model and sizes
    (L = 131072, D = 1536) with a single micro-perturbation dx = 1e-3 in one
    channel at t0 = 100000 and zero elsewhere.  Before t0 the tangent output
    is exactly zero in every channel (no background leakage); from t0 on
    every channel responds (the projections spread the pulse), and sampled
    channels, the perturbed one among them, match the oracle over the rest
    of the sequence."""
    t0, dp = 100000, 5
    inp = gu.custom("pulse128k")
    inp["dx"] = np.zeros_like(inp["dx"])
    inp["dx"][0, 0, t0, dp] = 1e-3
    print(f"case ghost pulse seg={seg}", flush=True)
    x, dx = gu.inputs_to_dev(inp)
    y, dy = binding.scan_jvp(x, dx, gu.params_to_dev(inp), seg_len=seg)
    torch.cuda.synchronize()
    leak = float(dy[:, :, :t0].abs().max())
    reach = bool(torch.all(dy[0, 0, t0:].abs().sum(0) > 0))
    ch = np.unique(np.concatenate([[0, dp, 1535], _channels(1536, 2, seed=17)]))
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, channels=ch, chunk=8192)
    idx = torch.from_numpy(ch).to(gu.dev())
    dys = dy.index_select(-1, idx)[:, :, t0:].cpu().numpy()
    e = gu.rel_l2(dys, dyo[:, :, t0:])
    print(f"ghost pulse seg={seg}: leak {leak:.1e}, every channel responds {reach}, rel_l2 dy after t0 {e:.3e} "
          f"on {len(ch)} channels", flush=True)
    if seg == 0:
        gu.record("ghost_pulse_t100000", {"t0": t0, "channel": dp, "magnitude": 1e-3, "leak_max_abs": leak,
                                          "every_channel_responds": reach, "dy_rel_l2_after_t0": e,
                                          "channels_compared": len(ch)})
    assert leak == 0.0 and reach
    assert e <= gu.TOL, e


def test_length_invariance():
    """The relative error against the oracle does not grow with L (App. B):
    the mamba130m recipe (dx ~ N(0,1)) at L = 2^10 .. 2^17 in the default
    plan, on 16 sampled channels; the fitted slope of the error in log2 L
    is recorded, and the error at the longest L stays within 3x of the
    shortest and below the bar."""
    Ls = [2 ** k for k in range(10, 18)]
    ch = _channels(1536, 2, seed=23)
    idx = torch.from_numpy(ch).to(gu.dev())
    base = gu.custom("mamba130m", seqlen=Ls[-1])
    prm = gu.params_to_dev(base)
    x_all, dx_all = gu.inputs_to_dev(base)
    yo, dyo, _, _ = oracle.scan_jvp(base["x"], base["dx"], base, channels=ch, chunk=8192)
    ey, edy = [], []
    for L in Ls:
        print(f"case length invariance L={L}", flush=True)
        y, dy = binding.scan_jvp(x_all[:, :L].contiguous(), dx_all[:, :, :L].contiguous(), prm)
        torch.cuda.synchronize()
        # the oracle is causal: its first L steps are the L-step call's outputs
        ey.append(gu.rel_l2(y.index_select(-1, idx).cpu().numpy(), yo[:, :L]))
        edy.append(gu.rel_l2(dy.index_select(-1, idx).cpu().numpy(), dyo[:, :, :L]))
    slope_y = float(np.polyfit(np.log2(Ls), ey, 1)[0])
    slope_dy = float(np.polyfit(np.log2(Ls), edy, 1)[0])
    print("L", Ls, "\nrel_l2 y", [f"{e:.2e}" for e in ey], "\nrel_l2 dy", [f"{e:.2e}" for e in edy],
          f"\nslope per doubling of L: y {slope_y:.2e}, dy {slope_dy:.2e}", flush=True)
    gu.record("length_invariance", {"L": Ls, "y_rel_l2": ey, "dy_rel_l2": edy, "slope_per_doubling_y": slope_y,
                                    "slope_per_doubling_dy": slope_dy, "channels_compared": len(ch)})
    assert max(ey + edy) <= gu.TOL
    assert ey[-1] <= 3 * ey[0] and edy[-1] <= 3 * edy[0], (ey, edy)
