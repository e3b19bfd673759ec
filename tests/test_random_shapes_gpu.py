"""Seeded random shapes and options against the fp64 oracle: every entry
point over batch sizes, channel counts and lengths that are not multiples of
anything (lengths 0 and 1 among them), every tiling override and, where the
kernels take them, the model variants.  Each case prints its draw before it
runs."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

SEGS = (0, -1, 16, 64, 256)
CHUNKS = (0, 1, 2, 5)


def _length(r, i):
    """Every eighth case takes one of the edge lengths 0, 1, 2, 17 in turn."""
    n = int(r.integers(3, 2500))
    return (0, 1, 2, 17)[(i // 8) % 4] if i % 8 == 0 else n


def _first_order_case(i):
    r = np.random.default_rng([4242, i])
    N = int(r.choice([4, 8, 16, 32, 64]))
    K = int(r.choice([1, 2, 4, 8]))
    kw = dict(seg_len=int(r.choice(SEGS)), chunk_segs=int(r.choice(CHUNKS)))
    base = str(r.choice(["mamba130m", "pulse128k", "stiff128k"]))
    cfg = dict(batch=int(r.integers(1, 4)), seqlen=_length(r, i), d_inner=int(r.integers(1, 301)), d_state=N,
               n_dirs=K, dx_kind="normal", in_dtype=str(r.choice(["f32", "bf16"])))
    extra = {}
    if N <= 16 and K <= 2:
        v = 1 if i % 8 == 3 else int(r.integers(0, 6))
        if v == 1:
            extra = dict(drive=str(r.choice(["euler", "zoh"])), act=str(r.choice(["identity", "silu"])), dres=True)
        elif v == 2:
            extra = dict(lowrank=int(r.integers(1, 65)))
        elif v == 3:
            extra = dict(complex=True)
            if r.integers(0, 2):
                extra.update(act="silu", dres=True)
            if r.integers(0, 2):
                extra.update(drive="zoh")
    elif i % 8 == 5:
        # the complex state with several threads per channel (N = 32, 64, or
        # four and eight directions)
        extra = dict(complex=True, drive="zoh" if i % 16 == 5 else "euler")
    return base, cfg, kw, extra


@pytest.mark.parametrize("i", range(96))
def test_random_first_order(i):
    base, cfg, kw, extra = _first_order_case(i)
    print(f"case first order #{i}: {base} {cfg} {kw} {extra}", flush=True)
    inp = gu.custom(base, **cfg)
    D, N = cfg["d_inner"], cfg["d_state"]
    r = np.random.default_rng([4243, i])
    if extra.get("dres"):
        inp["D_res"] = r.standard_normal(D).astype(np.float32)
    if extra.get("lowrank"):
        R = extra["lowrank"]
        inp["W_dx"] = (r.standard_normal((D, R)) / np.sqrt(D)).astype(np.float32)
        inp["W_dt"] = (r.uniform(-1.0, 1.0, (R, D)) / np.sqrt(R)).astype(np.float32)
    if extra.get("complex"):
        inp["A_im"] = (np.pi * r.uniform(0.1, 4.0, (D, N))).astype(np.float32)
    drive, act = extra.get("drive", "euler"), extra.get("act", "identity")
    y, dy, h, dh = gu.run(inp, drive=drive, act=act, return_state=True, **kw)
    yo, dyo, ho, dho = oracle.scan_jvp(inp["x"], inp["dx"], inp, drive=drive, act=act)
    if cfg["seqlen"] > 0:
        gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what=f"#{i}")
    for got, ref in ((h, ho), (dh, dho)):
        e = gu.rel_l2(got.cpu().numpy(), ref)
        assert e <= gu.TOL, (i, e)


@pytest.mark.parametrize("i", range(40))
def test_random_parameter_flows(i):
    r = np.random.default_rng([4244, i])
    N = int(r.choice([4, 8, 16]))
    cfg = dict(batch=int(r.integers(1, 4)), seqlen=_length(r, i), d_inner=int(r.integers(1, 301)), d_state=N,
               in_dtype=str(r.choice(["f32", "bf16"])))
    kw = dict(seg_len=int(r.choice(SEGS)), chunk_segs=int(r.choice(CHUNKS)),
              drive=str(r.choice(["euler", "zoh"])), act=str(r.choice(["identity", "silu"])),
              delta_params=bool(r.integers(0, 2)))
    dres = bool(r.integers(0, 2))
    print(f"case parameter flows #{i}: {cfg} {kw} dres={dres}", flush=True)
    inp = gu.custom("mamba130m", **cfg)
    inp["gy"] = inputs.make_adjoint(inp["cfg"])
    if dres:
        inp["D_res"] = r.standard_normal(cfg["d_inner"]).astype(np.float32)
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    out = binding.param_grads(x, gy, gu.params_to_dev(inp), return_state=True, **kw)
    torch.cuda.synchronize()
    yo, G, so = oracle.param_grads(inp["x"], inp["gy"], inp, drive=kw["drive"], act=kw["act"],
                                   delta_params=kw["delta_params"])
    ng = len(G)
    for k, (got, ref) in enumerate(zip(out[:1 + ng], (yo,) + tuple(G))):
        e = gu.rel_l2(got.cpu().numpy(), ref)
        assert e <= gu.TOL, (i, k, e)
    h, gam = out[1 + ng], out[2 + ng]
    assert gu.rel_l2(h.cpu().numpy(), so[0]) <= gu.TOL
    for k in range(len(so) - 1):
        assert gu.rel_l2(gam[k].cpu().numpy(), so[1 + k]) <= gu.TOL, (i, k)


@pytest.mark.parametrize("i", range(20))
def test_random_second_order(i):
    r = np.random.default_rng([4245, i])
    cfg = dict(batch=int(r.integers(1, 4)), seqlen=_length(r, i), d_inner=int(r.integers(1, 301)),
               d_state=int(r.choice([4, 8, 16])), n_dirs=2, dx_kind="normal")
    kw = dict(seg_len=int(r.choice(SEGS)), chunk_segs=int(r.choice(CHUNKS)))
    print(f"case second order #{i}: {cfg} {kw}", flush=True)
    inp = gu.custom("mamba130m", **cfg)
    x, dx = gu.inputs_to_dev(inp)
    y, dy, d2y = binding.scan_jvp2(x, dx, gu.params_to_dev(inp), **kw)
    torch.cuda.synchronize()
    (yo, yvo, ywo, yvwo), _ = oracle.scan_jvp2(inp["x"], inp["dx"][0], inp["dx"][1], inp)
    if cfg["seqlen"] > 0:
        gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, np.stack([yvo, ywo]), what=f"#{i}")
        assert gu.rel_l2(d2y.cpu().numpy(), yvwo) <= gu.TOL


@pytest.mark.parametrize("i", range(24))
def test_random_linear_attention(i):
    r = np.random.default_rng([4246, i])
    dk = int(r.choice([16, 32, 64]))
    cfg = inputs.LA_BY_NAME["la_tiny"].with_(batch=int(r.integers(1, 3)), heads=int(r.integers(1, 4)),
                                            seqlen=_length(r, i), d_key=dk, d_value=int(r.choice([64, 128, 192])),
                                            n_dirs=int(r.choice([1, 2])))
    kw = dict(seg_len=int(r.choice(SEGS)), chunk_segs=int(r.choice(CHUNKS)))
    print(f"case linear attention #{i}: {cfg} {kw}", flush=True)
    inp = inputs.make_la_inputs(cfg)
    names = ("q", "k", "v", "g", "dq", "dk", "dv", "dg")
    d = [torch.from_numpy(np.ascontiguousarray(inp[n])).to(gu.dev()) for n in names]
    o, do, S, dS = binding.la_scan_jvp(*d, return_state=True, **kw)
    torch.cuda.synchronize()
    oo, doo, So, dSo = oracle.la_scan_jvp(*[inp[n] for n in names])
    pairs = [(S, So), (dS, dSo)] + ([(o, oo), (do, doo)] if cfg.seqlen > 0 else [])
    for got, ref in pairs:
        e = gu.rel_l2(got.cpu().numpy(), ref)
        assert e <= gu.TOL, (i, e)
