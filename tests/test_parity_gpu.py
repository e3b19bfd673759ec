"""Parity of the HIP path (through the C ABI) with the fp64 oracle on seeded
inputs: element-by-element at sizes the oracle finishes in seconds, across
every tiling the planner can choose, ragged tiles, both evaluations
(sequential and segmented), both input dtypes and the stiff regime.  The
gate is a relative L2 error of 1e-5 per output (y and every dy_k)."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _check(inp, what, **kw):
    print(f"case {what}", flush=True)
    y, dy = gu.run(inp, **kw)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp)
    return gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what=what)


def test_tiny_workload_full():
    """B=1 L=1024 D=16 N=16 K=1, unit impulse tangent at t=0, d=0."""
    _check(inputs.make_inputs("tiny"), "tiny")


@pytest.mark.parametrize("seg", [0, -1, 64])
def test_multi_tile_ragged(seg):
    """Several channel blocks, segments and prefetch tiles, all ragged."""
    inp = gu.custom("mamba130m", batch=2, seqlen=1500, d_inner=300, n_dirs=2)
    _check(inp, f"ragged seg={seg}", seg_len=seg)


# Every (n_per_thread, n_split) the planner can choose, for K <= 2 and K >= 4;
# 605 steps end every evaluation on a partial tile of steps.
@pytest.mark.parametrize("N,K", [(4, 1), (8, 2), (16, 1), (32, 2), (64, 1),
                                 (4, 4), (8, 8), (16, 4), (32, 8), (64, 8)])
def test_tilings(N, K):
    inp = gu.custom("multidir", batch=1, seqlen=605, d_inner=72, d_state=N, n_dirs=K)
    p = binding.plan(1, 605, 72, N, K)
    _check(inp, f"N={N} K={K} nt={p['n_per_thread']} ns={p['n_split']}")


@pytest.mark.parametrize("N,K", [(16, 1), (64, 8)])
def test_sequential_evaluation(N, K):
    inp = gu.custom("multidir", batch=2, seqlen=700, d_inner=130, d_state=N, n_dirs=K)
    _check(inp, f"sequential N={N} K={K}", seg_len=-1, chunk_segs=0)


def test_bf16_stiff_regime():
    """bf16 inputs, A = -exp(U(0,7)), Delta in [1e-3, 10]: Abar underflows to
    zero in many lanes; no Inf/NaN and the same tolerance."""
    inp = gu.custom("stiff128k", seqlen=3000, d_inner=96)
    a = np.exp(np.logaddexp(0, inp["b_delta"].astype(np.float64))[:, None] * inp["A"])
    assert (a == 0).mean() > 0.05          # the regime really underflows
    _check(inp, "stiff bf16")
    _check(inp, "stiff bf16 sequential", seg_len=-1)


def test_biases_and_entry_state():
    inp = gu.custom("mamba130m", batch=2, seqlen=900, d_inner=64, n_dirs=2)
    g = np.random.default_rng(5)
    inp["b_B"] = g.standard_normal(16).astype(np.float32)
    inp["b_C"] = g.standard_normal(16).astype(np.float32)
    h0 = g.standard_normal((2, 64, 16)).astype(np.float32)
    dh0 = g.standard_normal((2, 2, 64, 16)).astype(np.float32)
    y, dy, h, dh = gu.run(inp, h_in=torch.from_numpy(h0), dh_in=torch.from_numpy(dh0), return_state=True)
    yo, dyo, ho, dho = oracle.scan_jvp(inp["x"], inp["dx"], inp, h_in=h0, dh_in=dh0)
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what="bias+state")
    assert gu.rel_l2(h.cpu().numpy(), ho) < 1e-5 and gu.rel_l2(dh.cpu().numpy(), dho) < 1e-5


@pytest.mark.parametrize("L", [1, 7, 255, 256, 257])
def test_short_sequences(L):
    inp = gu.custom("mamba130m", seqlen=L, d_inner=40, n_dirs=1)
    _check(inp, f"L={L}")


def test_empty_sequence_passes_state_through():
    inp = gu.custom("tiny", seqlen=0)
    g = np.random.default_rng(9)
    h0 = torch.from_numpy(g.standard_normal((1, 16, 16)).astype(np.float32))
    dh0 = torch.from_numpy(g.standard_normal((1, 1, 16, 16)).astype(np.float32))
    y, dy, h, dh = gu.run(inp, h_in=h0, dh_in=dh0, return_state=True)
    assert y.shape == (1, 0, 16) and dy.shape == (1, 1, 0, 16)
    assert torch.equal(h.cpu(), h0) and torch.equal(dh.cpu(), dh0)


def test_single_channel():
    inp = gu.custom("tiny", d_inner=1, seqlen=500, dx_kind="normal")
    _check(inp, "D=1")


def test_workspace_too_small_is_rejected():
    inp = gu.custom("tiny", seqlen=64)
    x, dx = gu.inputs_to_dev(inp)
    ws = torch.empty(16, device=gu.dev(), dtype=torch.uint8)
    nbytes = binding.workspace_bytes(1, 64, 16, 16, 1)
    assert nbytes > 16
    y = torch.full((1, 64, 16), 7.0, device=gu.dev())
    dy = torch.full((1, 1, 64, 16), 7.0, device=gu.dev())
    # a workspace tensor smaller than needed is replaced by the binding, so
    # call the ABI with a too-small size directly
    import ctypes
    pr = binding.make_params(1, 64, 16, 16, 1)
    prm = gu.params_to_dev(inp)
    for k in ("A", "w_delta", "b_delta", "W_B", "W_C"):
        setattr(pr, k, prm[k].data_ptr())
    pr.workspace, pr.workspace_bytes = ws.data_ptr(), 16
    rc = binding.lib().pgf_scan_jvp(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(dx.data_ptr()),
                                    ctypes.byref(pr), ctypes.c_void_p(y.data_ptr()),
                                    ctypes.c_void_p(dy.data_ptr()), None)
    assert rc == -3
    torch.cuda.synchronize()
    assert torch.all(y == 7.0) and torch.all(dy == 7.0)   # outputs untouched


@pytest.mark.parametrize("N,K,D", [(64, 2, 70), (32, 1, 37)])
def test_wide_f32_projection_ragged_channels(N, K, D):
    """f32 rows against 2N >= 64 columns take the split-plane projection;
    channel counts that are not multiples of 4 (scalar loads) and end in a
    partial 32-channel stage."""
    inp = gu.custom("multidir", batch=2, seqlen=500, d_inner=D, d_state=N, n_dirs=K)
    _check(inp, f"wide f32 N={N} K={K} D={D}")


def test_bf16_rows_match_f32_rows():
    """bf16 rows take their projections on the bf16 matrix cores with W cut
    into three bf16 planes (hi + mid + lo = W); the same values given as f32
    rows take the f32 matrix cores.  Both form exact products summed in f32,
    so the outputs agree to the rounding of the sums, far inside the oracle
    bar (a dropped plane, 2^-16 relative in B and C, would not)."""
    for N, D in ((16, 96), (64, 70)):
        inp = gu.custom("stiff128k", seqlen=1000, d_inner=D, d_state=N)
        y16, dy16 = gu.run(inp)
        y32, dy32 = gu.run(inp, bf16=False)
        ey = gu.rel_l2(y16.cpu().numpy(), y32.cpu().numpy())
        edy = gu.rel_l2(dy16.cpu().numpy(), dy32.cpu().numpy())
        print(f"bf16 rows vs f32 rows N={N} D={D}: y {ey:.2e} dy {edy:.2e}", flush=True)
        assert ey < 1e-6 and edy < 1e-6, (N, D, ey, edy)


@pytest.mark.parametrize("N,K,D", [(64, 8, 40), (32, 2, 98), (16, 4, 70), (8, 2, 64), (4, 1, 37)])
def test_bf16_multi_thread_channels(N, K, D):
    """bf16 inputs through the tilings where several threads share a channel,
    and through the narrow projections (2N = 8 and 16 columns), with channel
    counts that are not multiples of 4 (scalar load paths)."""
    inp = gu.custom("stiff128k", seqlen=900, d_inner=D, d_state=N, n_dirs=K)
    _check(inp, f"bf16 N={N} K={K} D={D}")


def test_timing_api_counts_launches():
    inp = gu.custom("mamba130m", seqlen=2000, d_inner=64, n_dirs=1)
    binding.timing_read()
    binding.timing_enable(True)
    try:
        gu.run(inp, seg_len=256, chunk_segs=3)
    finally:
        binding.timing_enable(False)
    t = binding.timing_read()
    # ceil(2000 / 768) = 3 host blocks: 3 x (projection, aggregate, carry,
    # output scan) plus the state import
    assert t["proj"][1] == 3 and t["seg_aggregate"][1] == 3 and t["carry"][1] == 3
    assert t["scan_out"][1] == 3 and t["state_io"][1] == 1
    assert all(ms >= 0 for ms, _ in t.values()) and t["scan_out"][0] > 0
    assert binding.timing_read()["scan_out"] == (0.0, 0)      # read clears


@pytest.mark.parametrize("in_dtype", ["f32", "bf16"])
def test_wide_channel_sum_splits(in_dtype):
    """D = 2112 > 2048: f32 projections cut the channel sum into two splits
    (2 x 1056 channels) and add them in order, bf16 ones take it whole;
    parity with the oracle, and bit-identical results for every host block
    size."""
    name = "stiff128k" if in_dtype == "bf16" else "mamba130m"
    inp = gu.custom(name, batch=1, seqlen=700, d_inner=2112, n_dirs=1)
    print(f"case wide D=2112 {in_dtype}", flush=True)
    y, dy = gu.run(inp, seg_len=64, chunk_segs=0)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp)
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what=f"wide D {in_dtype}")
    for cs in (1, 3):
        y2, dy2 = gu.run(inp, seg_len=64, chunk_segs=cs)
        assert torch.equal(y2, y) and torch.equal(dy2, dy), cs
