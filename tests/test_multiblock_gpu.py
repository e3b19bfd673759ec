"""The sequential evaluation across several host blocks (the block loop and
O(1) state hand-off of Alg. 1) for every entry point and model variant.

A sequential host block is chunk_segs * 4096 steps, so a call of 12 500
steps runs as four blocks at chunk_segs = 1, two at 2 and two at 3 (the
last block ragged each time).  Each case compares every channel with the
fp64 oracle and requires bit-identical outputs (and exported states) for
the three block sizes."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

L_MB = 12500          # > 3 * 4096: at least three host blocks at chunk_segs = 1
CHUNK_SEGS = (1, 2, 3)


def _plan_blocks(B, D, N, K, **kw):
    """Host blocks of the sequential plan for each chunk_segs (checked >= 3
    for chunk_segs = 1, so the test is not a single-block run)."""
    out = []
    for cs in CHUNK_SEGS:
        pl = binding.plan(B, L_MB, D, N, K, seg_len=-1, chunk_segs=cs, **kw)
        assert pl["seg_len"] == 0, pl
        out.append(pl["n_chunks"])
    print(f"sequential host blocks for chunk_segs {CHUNK_SEGS}: {out}", flush=True)
    assert out[0] >= 3, out
    return out


def _equal_all(runs, what):
    ref = runs[0]
    for cs, got in zip(CHUNK_SEGS[1:], runs[1:]):
        assert len(got) == len(ref)
        for i, (a, b) in enumerate(zip(got, ref)):
            assert torch.equal(a, b), (what, cs, i)


def _first_order(inp, what, D, N, K, drive="euler", act="identity", state=False, **plan_kw):
    print(f"case {what}", flush=True)
    _plan_blocks(1, D, N, K, drive=drive, act=act, **plan_kw)
    runs = [gu.run(inp, seg_len=-1, chunk_segs=cs, drive=drive, act=act, return_state=state) for cs in CHUNK_SEGS]
    _equal_all(runs, what)
    y, dy = runs[0][:2]
    yo, dyo, ho, dho = oracle.scan_jvp(inp["x"], inp["dx"], inp, drive=drive, act=act)
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what=what)
    if state:
        h, dh = runs[0][2:4]
        eh, edh = gu.rel_l2(h.cpu().numpy(), ho), gu.rel_l2(dh.cpu().numpy(), dho)
        print(f"{what} rel_l2 h_out={eh:.3e} dh_out={edh:.3e}", flush=True)
        assert eh <= gu.TOL and edh <= gu.TOL, (eh, edh)


@pytest.mark.parametrize("N,K", [(16, 1), (16, 2), (64, 8)])
def test_sequential_multiblock_first_order(N, K):
    D = 64
    inp = gu.custom("mamba130m" if K < 8 else "multidir", batch=1, seqlen=L_MB, d_inner=D, d_state=N, n_dirs=K)
    nt_ns = binding.plan(1, L_MB, D, N, K, seg_len=-1)
    print(f"tiling nt={nt_ns['n_per_thread']} ns={nt_ns['n_split']}", flush=True)
    _first_order(inp, f"multiblock N={N} K={K}", D, N, K, state=True)


def test_sequential_multiblock_bf16_stiff():
    inp = gu.custom("stiff128k", seqlen=L_MB, d_inner=64)
    _first_order(inp, "multiblock stiff bf16", 64, 16, 1, in_dtype="bf16")


def test_sequential_multiblock_split_call():
    """Two calls chained through the state at a host-block boundary equal
    one call bit for bit."""
    inp = gu.custom("mamba130m", batch=1, seqlen=L_MB, d_inner=64, n_dirs=2)
    y, dy, h, dh = gu.run(inp, seg_len=-1, chunk_segs=1, return_state=True)
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    s = 2 * 4096
    a = binding.scan_jvp(x[:, :s], dx[:, :, :s], prm, seg_len=-1, chunk_segs=1, return_state=True)
    b = binding.scan_jvp(x[:, s:], dx[:, :, s:], prm, seg_len=-1, chunk_segs=1, h_in=a[2], dh_in=a[3],
                         return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a[0], b[0]], 1), y) and torch.equal(torch.cat([a[1], b[1]], 2), dy)
    assert torch.equal(b[2], h) and torch.equal(b[3], dh)


def test_sequential_multiblock_variants():
    """ZOH drive + SiLU output map + residual weight."""
    inp = gu.custom("pulse128k", seqlen=L_MB, d_inner=64, dx_kind="normal", n_dirs=2)
    inp["D_res"] = np.random.default_rng(7).standard_normal(64).astype(np.float32)
    _first_order(inp, "multiblock zoh+silu+D_res", 64, 16, 2, drive="zoh", act="silu")


def test_sequential_multiblock_complex():
    inp = gu.custom("mamba130m", batch=1, seqlen=L_MB, d_inner=64, n_dirs=2)
    r = np.random.default_rng(9)
    inp["A_im"] = (np.pi * r.uniform(0.1, 4.0, (64, 16)) * r.choice([-1, 1], (64, 16))).astype(np.float32)
    print("case multiblock complex", flush=True)
    _plan_blocks(1, 64, 16, 2, complex_a=True)
    runs = [gu.run(inp, seg_len=-1, chunk_segs=cs, return_state=True) for cs in CHUNK_SEGS]
    _equal_all(runs, "complex")
    y, dy, h, dh = runs[0]
    yo, dyo, ho, dho = oracle.scan_jvp(inp["x"], inp["dx"], inp)
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what="multiblock complex")
    # both parts of the complex state against the oracle
    for got, ref in ((h, ho), (dh, dho)):
        e = gu.rel_l2(got.cpu().numpy(), ref)
        print(f"multiblock complex state rel_l2 {e:.3e}", flush=True)
        assert e <= gu.TOL, e


def test_sequential_multiblock_groups():
    D, G = 128, 2
    inp = gu.custom("mamba130m", batch=1, seqlen=L_MB, d_inner=D, n_dirs=1)
    r = np.random.default_rng(11)
    inp["n_groups"] = G
    inp["W_B"] = (r.standard_normal((D, G * 16)) / np.sqrt(D)).astype(np.float32)
    inp["W_C"] = (r.standard_normal((D, G * 16)) / np.sqrt(D)).astype(np.float32)
    _first_order(inp, "multiblock groups", D, 16, 1, groups=G)


def test_sequential_multiblock_low_rank():
    D, R = 64, 16
    inp = gu.custom("mamba130m", batch=1, seqlen=L_MB, d_inner=D, n_dirs=2)
    r = np.random.default_rng(13)
    inp["W_dx"] = (r.standard_normal((D, R)) / np.sqrt(D)).astype(np.float32)
    inp["W_dt"] = (r.uniform(-1.0, 1.0, (R, D)) / np.sqrt(R)).astype(np.float32)
    _first_order(inp, "multiblock low rank", D, 16, 2, dt_rank=R)


def test_sequential_multiblock_second_order():
    inp = gu.custom("mamba130m", batch=1, seqlen=L_MB, d_inner=64, n_dirs=2)
    print("case multiblock order 2", flush=True)
    _plan_blocks(1, 64, 16, 2, order=2)
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    runs = []
    for cs in CHUNK_SEGS:
        runs.append(binding.scan_jvp2(x, dx, prm, seg_len=-1, chunk_segs=cs, return_state=True))
        torch.cuda.synchronize()
    _equal_all(runs, "order 2")
    y, dy, d2y = runs[0][:3]
    (yo, yvo, ywo, yvwo), _ = oracle.scan_jvp2(inp["x"], inp["dx"][0], inp["dx"][1], inp)
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, np.stack([yvo, ywo]), what="multiblock order 2")
    e = gu.rel_l2(d2y.cpu().numpy(), yvwo)
    print(f"multiblock order 2 rel_l2 d2y={e:.3e}", flush=True)
    assert e <= gu.TOL, e


@pytest.mark.parametrize("drive,omap,dlt", [("euler", False, False), ("zoh", False, False), ("euler", True, False),
                                            ("zoh", True, False), ("euler", False, True), ("zoh", True, True)])
def test_sequential_multiblock_param_grads(drive, omap, dlt):
    """omap: SiLU output map with a residual weight (its gradient too);
    dlt: the flows of the step size's parameters."""
    inp = gu.custom("mamba130m", batch=1, seqlen=L_MB, d_inner=64)
    inp["gy"] = inputs.make_adjoint(inp["cfg"])
    act = "silu" if omap else "identity"
    if omap:
        inp["D_res"] = np.random.default_rng(15).standard_normal(64).astype(np.float32)
    print(f"case multiblock parameter flows {drive} act={act}", flush=True)
    _plan_blocks(1, 64, 16, 1, order=3, drive=drive, act=act, delta_flows=dlt)
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    prm = gu.params_to_dev(inp)
    runs = []
    for cs in CHUNK_SEGS:
        runs.append(binding.param_grads(x, gy, prm, seg_len=-1, chunk_segs=cs, return_state=True, drive=drive,
                                        act=act, delta_params=dlt))
        torch.cuda.synchronize()
    _equal_all(runs, "parameter flows")
    ng = (4 if omap else 3) + (2 if dlt else 0)
    got = runs[0][:1 + ng]
    yo, G, _ = oracle.param_grads(inp["x"], inp["gy"], inp, drive=drive, act=act, delta_params=dlt)
    errs = [gu.rel_l2(a.cpu().numpy(), b) for a, b in zip(got, (yo,) + tuple(G))]
    print("multiblock param rel_l2 " + " ".join(f"{e:.3e}" for e in errs), flush=True)
    assert len(errs) == 1 + ng and max(errs) <= gu.TOL, errs


def test_sequential_multiblock_linear_attention():
    cfg = inputs.LA_BY_NAME["la_tiny"].with_(batch=1, heads=2, seqlen=L_MB, d_key=32, n_dirs=1)
    inp = inputs.make_la_inputs(cfg)
    names = ("q", "k", "v", "g", "dq", "dk", "dv", "dg")
    print("case multiblock linear attention", flush=True)
    blocks = []
    for cs in CHUNK_SEGS:
        pl = binding.la_plan(1, 2, L_MB, 32, cfg.d_value, 1, seg_len=-1, chunk_segs=cs)
        assert pl["seg_len"] == 0
        blocks.append(pl["n_chunks"])
    print(f"sequential host blocks {blocks}", flush=True)
    assert blocks[0] >= 3
    d = [torch.from_numpy(np.ascontiguousarray(inp[n])).to(gu.dev()) for n in names]
    runs = []
    for cs in CHUNK_SEGS:
        runs.append(binding.la_scan_jvp(*d, seg_len=-1, chunk_segs=cs, return_state=True))
        torch.cuda.synchronize()
    _equal_all(runs, "linear attention")
    o, do, S, dS = runs[0]
    oo, doo, So, dSo = oracle.la_scan_jvp(*[inp[n] for n in names])
    for got, ref, nm in ((o, oo, "o"), (do, doo, "do"), (S, So, "S"), (dS, dSo, "dS")):
        e = gu.rel_l2(got.cpu().numpy(), ref)
        print(f"multiblock la rel_l2 {nm}={e:.3e}", flush=True)
        assert e <= gu.TOL, (nm, e)
