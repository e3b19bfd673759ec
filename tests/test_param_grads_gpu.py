"""Parameter flows (App. E, Alg. 2) on the GPU against the fp64 oracle: the
primal y and the accumulated gradients dl/dA and of the per-lane offsets of
B and C for a seeded adjoint signal; y bit-identical to pgf_scan_jvp;
gradients bit-identical for every host block size; split calls chained
through the state; accumulation into caller buffers; argument checks."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _case(name, **kw):
    inp = gu.custom(name, **kw)
    inp["gy"] = inputs.make_adjoint(inp["cfg"])
    return inp


def _run(inp, **kw):
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    out = binding.param_grads(x, gy, gu.params_to_dev(inp), **kw)
    torch.cuda.synchronize()
    return out


def _block_channels(D, g, block=64):
    """One seeded channel of every 64-channel block and the first and last."""
    picks = [int(g.integers(s, min(s + block, D))) for s in range(0, D, block)]
    return np.unique(np.concatenate([[0, D - 1], picks])).astype(np.int64)


def _check(inp, what, channels=None, scaled=False, record=None, **kw):
    """y and every gradient (dl/dD_res too when inp has D_res) against the
    oracle, optionally on sampled channels only.  scaled: measure the step
    size's gradients against the sums of the absolute values of their terms
    (see gpu_util.sum_error) instead of their own norms.  record: key of the
    errors in the parity record."""
    print(f"case {what}", flush=True)
    dlt = kw.get("delta_params", False)
    ng = (4 if inp.get("D_res") is not None else 3) + (2 if dlt else 0)
    got = list(_run(inp, **kw)[:1 + ng])
    out = oracle.param_grads(inp["x"], inp["gy"], inp, channels=channels, chunk=None if channels is None else 8192,
                             drive=kw.get("drive", "euler"), act=kw.get("act", "identity"), delta_params=dlt,
                             return_scale=dlt and scaled)
    yo, G = out[0], out[1]
    assert len(G) == ng
    if channels is not None:
        idx = torch.from_numpy(np.asarray(channels)).to(gu.dev())
        got = [got[0].index_select(-1, idx)] + [g.index_select(0, idx) for g in got[1:]]
    errs = [gu.rel_l2(a.cpu().numpy(), b) for a, b in zip(got, (yo,) + tuple(G))]
    if dlt and scaled:
        # dl/dw_delta and dl/db_delta are sums of terms of both signs over
        # every step: over long sequences their error is measured against the
        # sum of the terms' absolute values (the plain measure is printed too)
        plain = errs[-2:]
        errs[-2:] = [gu.sum_error(got[-2 + i].cpu().numpy(), G[-2 + i], out[3][i]) for i in range(2)]
        print(f"{what} plain rel_l2 gW={plain[0]:.3e} gS={plain[1]:.3e}", flush=True)
    names = ("y", "gA", "gB", "gC") + (("gD",) if inp.get("D_res") is not None else ()) + ("gW", "gS")
    print(f"{what} rel_l2 " + " ".join(f"{n}={e:.3e}" for n, e in zip(names, errs)), flush=True)
    if record:
        rec = {f"{n}_rel_l2": float(e) for n, e in zip(names, errs)}
        rec["channels_compared"] = int(len(channels)) if channels is not None else int(inp["x"].shape[-1])
        if dlt and scaled:
            rec["step_size_gradient_measure"] = "error / sum of the absolute values of the terms"
        gu.record(record, rec)
    for a in got:
        assert torch.all(torch.isfinite(a))
    assert max(errs) <= gu.TOL, (what, errs)


@pytest.mark.parametrize("N,seg", [(16, 0), (8, 0), (4, 0), (16, -1), (16, 64), (32, 0), (64, 64), (32, -1)])
def test_param_grads_parity(N, seg):
    inp = _case("mamba130m", batch=2, seqlen=1100, d_inner=70, d_state=N)
    _check(inp, f"param N={N} seg={seg}", seg_len=seg)


def test_param_grads_bf16_stiff():
    _check(_case("stiff128k", seqlen=1500, d_inner=64), "param stiff bf16")


def test_param_grads_full_size_sampled_channels():
    """pulse128k's sizes (B=1, L=131072, D=1536, N=16) in the default plan,
    against the oracle over the whole sequence on one channel of every
    64-channel block."""
    inp = _case("pulse128k")
    g = np.random.default_rng(5)
    ch = _block_channels(1536, g)
    _check(inp, "param pulse128k full", channels=ch, record="param_pulse128k")


def test_primal_matches_pgf_scan_jvp():
    inp = _case("mamba130m", batch=1, seqlen=900, d_inner=96)
    for seg in (128, -1):
        y = _run(inp, seg_len=seg, chunk_segs=4)[0]
        y1, _ = gu.run(inp, seg_len=seg, chunk_segs=4)
        assert torch.equal(y, y1), seg


def test_block_invariance_and_handoff():
    inp = _case("mamba130m", batch=2, seqlen=1000, d_inner=48)
    ref = _run(inp, seg_len=64, chunk_segs=1, return_state=True)
    for cs in (3, 0):
        got = _run(inp, seg_len=64, chunk_segs=cs, return_state=True)
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    prm = gu.params_to_dev(inp)
    s = 384
    a = binding.param_grads(x[:, :s], gy[:, :s], prm, seg_len=64, return_state=True)
    b = binding.param_grads(x[:, s:], gy[:, s:], prm, seg_len=64, h_in=a[4], gamma_in=a[5], grads=a[1:4],
                            return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a[0], b[0]], 1), ref[0])
    assert torch.equal(b[4], ref[4]) and torch.equal(b[5], ref[5])
    for i in (1, 2, 3):   # the split adds the two halves' sums: rounding only
        assert gu.rel_l2(b[i].cpu().numpy(), ref[i].cpu().numpy()) < 1e-6, i


def test_entry_state_matches_oracle():
    inp = _case("mamba130m", batch=1, seqlen=700, d_inner=40)
    g = np.random.default_rng(41)
    st = [g.standard_normal((1, 40, 16)).astype(np.float32) for _ in range(3)]
    y, gA, gB, gC, h, gam = _run(inp, h_in=torch.from_numpy(st[0]), gamma_in=torch.from_numpy(np.stack(st[1:])),
                                 return_state=True)
    yo, G, so = oracle.param_grads(inp["x"], inp["gy"], inp, state=tuple(st))
    for got, ref in ((y, yo), (gA, G[0]), (gB, G[1]), (gC, G[2]), (h, so[0]), (gam[0], so[1]), (gam[1], so[2])):
        assert gu.rel_l2(got.cpu().numpy(), ref) < gu.TOL


def test_gradients_are_added_to_the_callers_buffers():
    inp = _case("mamba130m", batch=1, seqlen=500, d_inner=32)
    _, gA, gB, gC = _run(inp)
    pre = tuple(torch.full_like(g, 0.25) for g in (gA, gB, gC))
    _, hA, hB, hC = _run(inp, grads=pre)
    for g, h in ((gA, hA), (gB, hB), (gC, hC)):
        assert torch.allclose(h, g + 0.25, rtol=1e-6, atol=1e-6)
    # an empty sequence adds nothing and passes the state through
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    h0 = torch.randn(1, 32, 16, device=gu.dev())
    out = binding.param_grads(x[:, :0], gy[:, :0], gu.params_to_dev(inp), h_in=h0, grads=pre, return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(out[1], pre[0]) and torch.equal(out[4], h0) and torch.all(out[5] == 0)


def test_zero_adjoint_gives_zero_gradients():
    inp = _case("mamba130m", batch=1, seqlen=300, d_inner=32)
    inp["gy"][:] = 0.0
    _, gA, gB, gC = _run(inp)
    assert all(torch.all(g == 0) for g in (gA, gB, gC))


def test_argument_checks():
    inp = _case("tiny", seqlen=64)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        binding.plan(1, 64, 16, 32, 1, order=3, complex_a=True)
    pr = binding.make_params(1, 64, 16, 16, 1, order=1)
    lib = binding.lib()
    assert lib.pgf_param_grads(None, None, ctypes.byref(pr), None, None, None, None, None) == -1
    x, _ = gu.inputs_to_dev(inp)
    with pytest.raises(ValueError, match="float32"):
        binding.param_grads(x, torch.zeros_like(x, dtype=torch.bfloat16), gu.params_to_dev(inp))
    gy = torch.zeros_like(x)
    with pytest.raises(ValueError, match="grads"):
        binding.param_grads(x, gy, gu.params_to_dev(inp), grads=(torch.zeros(16, 16, device=gu.dev()),) * 2
                            + (torch.zeros(16, 8, device=gu.dev()),))


# ------------------------------------------------------------ zero-order-hold drive
# GammaA gains the drive's derivative in A: (Delta Abar - e)/A * B x, from a
# series for |Delta A| < 1/4 and from the closed form above.

@pytest.mark.parametrize("N,seg", [(16, 0), (8, -1), (4, 64), (16, -1), (64, -1), (32, 64)])
def test_param_grads_zoh_parity(N, seg):
    inp = _case("mamba130m", batch=2, seqlen=1100, d_inner=70, d_state=N)
    _check(inp, f"param zoh N={N} seg={seg}", seg_len=seg, drive="zoh")


def test_param_grads_zoh_small_steps_and_stiff():
    """Delta A on both sides of the series / closed-form switch: pulse128k's
    Delta in [1e-4, 1e-2] (series) and the stiff bf16 workload."""
    _check(_case("pulse128k", seqlen=2000, d_inner=64), "param zoh small steps", drive="zoh")
    _check(_case("stiff128k", seqlen=1500, d_inner=64), "param zoh stiff bf16", drive="zoh")


def test_param_grads_zoh_block_invariance_and_handoff():
    inp = _case("mamba130m", batch=2, seqlen=1000, d_inner=48)
    ref = _run(inp, seg_len=64, chunk_segs=1, return_state=True, drive="zoh")
    for cs in (3, 0):
        got = _run(inp, seg_len=64, chunk_segs=cs, return_state=True, drive="zoh")
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs
    # the Euler flows differ: the drive's A-dependence reached the gradient
    eul = _run(inp, seg_len=64, chunk_segs=1)
    assert not torch.equal(eul[1], ref[1]) and torch.equal(eul[2], eul[2])


def test_param_grads_zoh_full_size_sampled_channels():
    inp = _case("pulse128k")
    g = np.random.default_rng(6)
    ch = _block_channels(1536, g)
    _check(inp, "param zoh pulse128k full", channels=ch, drive="zoh", record="param_pulse128k_zoh")


# ------------------------------------------------------------ output map
# y = act(sum_n C h + D_res x): the sums take w = gy act'(yhat) in place of
# gy, and dl/dD_res = sum w x is returned as a fourth gradient.

def _with_dres(inp, seed=17):
    inp["D_res"] = np.random.default_rng(seed).standard_normal(inp["x"].shape[-1]).astype(np.float32)
    return inp


@pytest.mark.parametrize("act,dres,drive,N,seg", [
    ("silu", True, "euler", 16, 0), ("silu", False, "euler", 8, -1), ("identity", True, "zoh", 16, 64),
    ("silu", True, "zoh", 4, -1), ("silu", True, "euler", 16, -1), ("silu", True, "zoh", 16, 0),
    ("silu", True, "euler", 64, 0), ("silu", True, "zoh", 32, -1)])
def test_param_grads_output_map_parity(act, dres, drive, N, seg):
    inp = _case("mamba130m", batch=2, seqlen=1100, d_inner=70, d_state=N)
    if dres:
        _with_dres(inp)
    _check(inp, f"param map act={act} dres={dres} {drive} N={N} seg={seg}", seg_len=seg, drive=drive, act=act)


def test_param_grads_output_map_bf16_stiff():
    _check(_with_dres(_case("stiff128k", seqlen=1500, d_inner=64)), "param map stiff bf16", act="silu")


def test_param_grads_output_map_primal_and_blocks():
    """y equals pgf_scan_jvp's with the same output map bit for bit; every
    output (dl/dD_res included) is bit-identical for every host block size;
    a split call chained through the state, adding into the same four
    buffers, matches one call up to the rounding of the additions."""
    inp = _with_dres(_case("mamba130m", batch=2, seqlen=1000, d_inner=48))
    for seg in (64, -1):
        y = _run(inp, seg_len=seg, chunk_segs=4, act="silu")[0]
        y1, _ = gu.run(inp, seg_len=seg, chunk_segs=4, act="silu")
        assert torch.equal(y, y1), seg
    ref = _run(inp, seg_len=64, chunk_segs=1, return_state=True, act="silu")
    assert len(ref) == 7
    for cs in (3, 0):
        got = _run(inp, seg_len=64, chunk_segs=cs, return_state=True, act="silu")
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    prm = gu.params_to_dev(inp)
    s = 384
    a = binding.param_grads(x[:, :s], gy[:, :s], prm, seg_len=64, return_state=True, act="silu")
    b = binding.param_grads(x[:, s:], gy[:, s:], prm, seg_len=64, h_in=a[5], gamma_in=a[6], grads=a[1:5],
                            return_state=True, act="silu")
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a[0], b[0]], 1), ref[0])
    assert torch.equal(b[5], ref[5]) and torch.equal(b[6], ref[6])
    for i in (1, 2, 3, 4):
        assert gu.rel_l2(b[i].cpu().numpy(), ref[i].cpu().numpy()) < 1e-6, i


def test_param_grads_output_map_identity_residual():
    """Identity map with D_res: the flows of A, B, C are those without the
    residual weight bit for bit (only y changes), and dl/dD_res equals
    sum over b and t of gy x (the closed form), to rounding."""
    inp = _case("mamba130m", batch=2, seqlen=800, d_inner=64)
    base = _run(inp, seg_len=128)
    got = _run(_with_dres(inp), seg_len=128)
    for i in (1, 2, 3):
        assert torch.equal(got[i], base[i]), i
    ref = (inp["gy"].astype(np.float64) * inp["x"].astype(np.float64)).sum((0, 1))
    assert gu.rel_l2(got[4].cpu().numpy(), ref) < 1e-6


def test_param_grads_output_map_full_size_sampled_channels():
    inp = _with_dres(_case("pulse128k"))
    g = np.random.default_rng(7)
    ch = _block_channels(1536, g)
    _check(inp, "param map pulse128k full", channels=ch, act="silu", record="param_pulse128k_silu_dres")


def test_param_grads_output_map_argument_checks():
    inp = _with_dres(_case("tiny", seqlen=64))
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.zeros_like(x)
    prm = gu.params_to_dev(inp)
    D, N = inp["A"].shape
    with pytest.raises(ValueError, match="grads"):   # three buffers where D_res needs four
        binding.param_grads(x, gy, prm, grads=tuple(torch.zeros(D, N, device=gu.dev()) for _ in range(3)))
    # through the C-ABI: D_res set and grad_D_res NULL
    pr = binding.make_params(1, 64, D, N, 1, order=3, act="silu")
    keep = []
    binding._model_params(pr, prm, D, gu.dev(), keep)
    pr.D_res = prm["D_res"].data_ptr()
    ws = torch.empty(binding.workspace_bytes(1, 64, D, N, 1, order=3, act="silu"), dtype=torch.uint8,
                     device=gu.dev())
    pr.workspace, pr.workspace_bytes = ws.data_ptr(), ws.numel()
    y = torch.empty_like(x)
    g3 = [torch.zeros(D, N, device=gu.dev()) for _ in range(3)]
    rc = binding.lib().pgf_param_grads(x.data_ptr(), gy.data_ptr(), ctypes.byref(pr), y.data_ptr(),
                                       *[g.data_ptr() for g in g3], None)
    assert rc == -1   # PGF_ERR_INVALID_ARG


def test_param_grads_zoh_zero_eigenvalues():
    """Columns of A exactly 0 with the ZOH drive: e and de/dA take their
    limits Delta and Delta^2/2 (the closed forms' 1/A must not leak)."""
    inp = _case("mamba130m", batch=1, seqlen=1000, d_inner=64)
    inp["A"] = inp["A"].copy()
    inp["A"][:, [0, 9]] = 0.0
    for seg in (64, -1):
        _check(inp, f"param zoh zero eigenvalues seg={seg}", seg_len=seg, drive="zoh")



# ------------------------------------------------------------ step-size parameters
# delta_params: the flows of w_delta and b_delta (Delta = softplus(w x + b))
# beside the others, with dl/dw_delta and dl/db_delta per channel.

@pytest.mark.parametrize("drive,act,dres,N,seg", [
    ("euler", "identity", False, 16, 0), ("euler", "identity", False, 8, -1), ("zoh", "identity", False, 16, 64),
    ("euler", "silu", True, 16, -1), ("zoh", "silu", True, 16, 0), ("zoh", "silu", True, 4, -1),
    ("euler", "identity", False, 64, 64), ("zoh", "silu", True, 32, 0), ("euler", "silu", True, 64, -1)])
def test_param_grads_step_size_parity(drive, act, dres, N, seg):
    inp = _case("mamba130m", batch=2, seqlen=1100, d_inner=70, d_state=N)
    if dres:
        _with_dres(inp)
    _check(inp, f"param step size {drive} act={act} dres={dres} N={N} seg={seg}", seg_len=seg, drive=drive,
           act=act, delta_params=True)


def test_param_grads_step_size_bf16_stiff():
    _check(_case("stiff128k", seqlen=1500, d_inner=64), "param step size stiff bf16", delta_params=True)


def test_param_grads_step_size_leaves_the_rest_unchanged():
    """The other outputs are the same bits with and without the step size's
    flows (the same arithmetic runs for them)."""
    inp = _with_dres(_case("mamba130m", batch=2, seqlen=900, d_inner=64))
    for drive, seg in (("euler", 64), ("zoh", -1)):
        a = _run(inp, seg_len=seg, drive=drive, act="silu", return_state=True)
        b = _run(inp, seg_len=seg, drive=drive, act="silu", return_state=True, delta_params=True)
        for i in range(5):
            assert torch.equal(a[i], b[i]), (drive, i)
        assert torch.equal(a[5], b[7]) and torch.equal(a[6], b[8][:2]), drive


def test_param_grads_step_size_blocks_and_handoff():
    inp = _case("mamba130m", batch=2, seqlen=1000, d_inner=48)
    ref = _run(inp, seg_len=64, chunk_segs=1, return_state=True, delta_params=True)
    assert len(ref) == 8 and tuple(ref[7].shape) == (4, 2, 48, 16)
    for cs in (3, 0):
        got = _run(inp, seg_len=64, chunk_segs=cs, return_state=True, delta_params=True)
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    prm = gu.params_to_dev(inp)
    s = 384
    a = binding.param_grads(x[:, :s], gy[:, :s], prm, seg_len=64, return_state=True, delta_params=True)
    b = binding.param_grads(x[:, s:], gy[:, s:], prm, seg_len=64, h_in=a[6], gamma_in=a[7], grads=a[1:6],
                            return_state=True, delta_params=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a[0], b[0]], 1), ref[0])
    assert torch.equal(b[6], ref[6]) and torch.equal(b[7], ref[7])
    for i in range(1, 6):
        assert gu.rel_l2(b[i].cpu().numpy(), ref[i].cpu().numpy()) < 1e-6, i
    # the entry state of all five planes against the oracle
    g = np.random.default_rng(19)
    st = [g.standard_normal((2, 48, 16)).astype(np.float32) for _ in range(5)]
    got = _run(inp, h_in=torch.from_numpy(st[0]), gamma_in=torch.from_numpy(np.stack(st[1:])), return_state=True,
               delta_params=True)
    yo, G, so = oracle.param_grads(inp["x"], inp["gy"], inp, state=tuple(st), delta_params=True)
    for i, (gt, rf) in enumerate(zip(got[:6], (yo,) + tuple(G))):
        assert gu.rel_l2(gt.cpu().numpy(), rf) < gu.TOL, i
    assert gu.rel_l2(got[6].cpu().numpy(), so[0]) < gu.TOL
    for k in range(4):
        assert gu.rel_l2(got[7][k].cpu().numpy(), so[1 + k]) < gu.TOL, k


def test_param_grads_step_size_full_size_sampled_channels():
    inp = _with_dres(_case("pulse128k"))
    g = np.random.default_rng(8)
    ch = _block_channels(1536, g)
    _check(inp, "param step size pulse128k full", channels=ch, act="silu", delta_params=True, scaled=True,
           record="param_pulse128k_step_size")


def test_param_grads_step_size_argument_checks():
    inp = _case("tiny", seqlen=64)
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.zeros_like(x)
    prm = gu.params_to_dev(inp)
    D, N = inp["A"].shape
    with pytest.raises(ValueError, match="grads"):   # three buffers where five are needed
        binding.param_grads(x, gy, prm, grads=tuple(torch.zeros(D, N, device=gu.dev()) for _ in range(3)),
                            delta_params=True)
    with pytest.raises(RuntimeError, match="INVALID_ARG"):   # the flag belongs to the parameter flows
        binding.plan(1, 64, D, N, 1, order=1, delta_flows=True)
    # through the C-ABI: the flag set and grad_b_delta NULL
    pr = binding.make_params(1, 64, D, N, 1, order=3, delta_flows=True)
    keep = []
    binding._model_params(pr, prm, D, gu.dev(), keep)
    ws = torch.empty(binding.workspace_bytes(1, 64, D, N, 1, order=3, delta_flows=True), dtype=torch.uint8,
                     device=gu.dev())
    pr.workspace, pr.workspace_bytes = ws.data_ptr(), ws.numel()
    gw = torch.zeros(D, device=gu.dev())
    pr.grad_w_delta = gw.data_ptr()
    y = torch.empty_like(x)
    g3 = [torch.zeros(D, N, device=gu.dev()) for _ in range(3)]
    rc = binding.lib().pgf_param_grads(x.data_ptr(), gy.data_ptr(), ctypes.byref(pr), y.data_ptr(),
                                       *[g.data_ptr() for g in g3], None)
    assert rc == -1   # PGF_ERR_INVALID_ARG
