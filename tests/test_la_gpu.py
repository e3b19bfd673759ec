"""Decaying linear attention with its tangent flow (App. F) on the GPU
against the fp64 oracle: several key sizes, one and two directions, the
segmented and sequential evaluations, ragged lengths, the full rwkv128k
size on sampled heads, bit-identical results for every host block size and
for split calls chained through the state, and argument checks."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu
NAMES = ("q", "k", "v", "g", "dq", "dk", "dv", "dg")


def _case(name="la_tiny", **kw):
    cfg = inputs.LA_BY_NAME[name].with_(**kw)
    return inputs.make_la_inputs(cfg)


def _dev(inp, heads=None):
    out = []
    for n in NAMES:
        a = inp[n]
        if heads is not None:
            a = a[..., heads, :, :]
        out.append(torch.from_numpy(np.ascontiguousarray(a)).to(gu.dev()))
    return out


def _run(inp, **kw):
    out = binding.la_scan_jvp(*_dev(inp), **kw)
    torch.cuda.synchronize()
    return out


def _check(inp, what, **kw):
    print(f"case {what}", flush=True)
    o, do = _run(inp, **kw)[:2]
    oo, doo, _, _ = oracle.la_scan_jvp(*[inp[n] for n in NAMES])
    e1, e2 = gu.rel_l2(o.cpu().numpy(), oo), gu.rel_l2(do.cpu().numpy(), doo)
    print(f"{what} rel_l2 o={e1:.3e} do={e2:.3e}", flush=True)
    assert torch.all(torch.isfinite(o)) and torch.all(torch.isfinite(do))
    assert e1 <= gu.TOL and e2 <= gu.TOL, (what, e1, e2)


@pytest.mark.parametrize("DK,K,seg", [(16, 1, 0), (32, 1, 0), (64, 1, 0), (64, 2, 0), (16, 2, -1), (64, 1, -1),
                                      (32, 1, 64)])
def test_la_parity(DK, K, seg):
    inp = _case(batch=2, heads=3, seqlen=1100, d_key=DK, n_dirs=K)
    _check(inp, f"la DK={DK} K={K} seg={seg}", seg_len=seg)


def test_la_wide_values_and_constant_decay():
    inp = _case(heads=2, seqlen=700, d_key=32, d_value=128)
    _check(inp, "la DV=128")
    # RetNet: one constant decay per head
    inp = _case(heads=2, seqlen=900, d_key=16)
    gam = np.log(np.array([0.97, 0.995], dtype=np.float32))
    inp["g"][:] = gam[None, :, None, None]
    _check(inp, "la retnet decay")


@pytest.mark.parametrize("seg", [0, -1])
def test_la_degenerate_decays(seg):
    """No decay (g = 0: the linear transformer, every segment transition 1,
    the state only grows) and a decay that underflows (g = -200: alpha is 0
    in f32, so S_t = k_t v_t^T and o_t = (q_t . k_t) v_t) in two heads of
    one call, with tangents of g zero in the first and N(0,1) in the
    second."""
    inp = _case(heads=2, seqlen=1100, d_key=32)
    inp["g"][:, 0] = 0.0
    inp["dg"][:, :, 0] = 0.0
    inp["g"][:, 1] = -200.0
    _check(inp, f"la degenerate decays seg={seg}", seg_len=seg)


def test_la_full_size_sampled_heads():
    """rwkv128k (B=1, H=32, L=131072, dk=dv=64) in the default plan; heads are
    independent, so the oracle runs on three of them."""
    inp = _case("rwkv128k")
    print("case rwkv128k full: GPU", flush=True)
    o, do = _run(inp)
    heads = [0, 17, 31]
    og = o[:, heads].cpu().numpy()
    dog = do[:, :, heads].cpu().numpy()
    del o, do
    torch.cuda.empty_cache()
    print(f"case rwkv128k full: oracle on heads {heads}", flush=True)
    sub = [np.ascontiguousarray(inp[n][..., heads, :, :]) for n in NAMES]
    oo, doo, _, _ = oracle.la_scan_jvp(*sub, chunk=16384)
    e1, e2 = gu.rel_l2(og, oo), gu.rel_l2(dog, doo)
    print(f"rwkv128k rel_l2 o={e1:.3e} do={e2:.3e}", flush=True)
    gu.record("rwkv128k", {"heads_compared": heads, "o_rel_l2": e1, "do_rel_l2": e2})
    assert e1 <= gu.TOL and e2 <= gu.TOL


def test_la_block_invariance_and_handoff():
    inp = _case(batch=2, heads=2, seqlen=1000, d_key=32, n_dirs=2)
    ref = _run(inp, seg_len=64, chunk_segs=1, return_state=True)
    for cs in (3, 0):
        got = _run(inp, seg_len=64, chunk_segs=cs, return_state=True)
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs
    d = _dev(inp)
    s = 384
    first = binding.la_scan_jvp(*[t[..., :s, :] for t in d], seg_len=64, return_state=True)
    second = binding.la_scan_jvp(*[t[..., s:, :] for t in d], seg_len=64, S_in=first[2], dS_in=first[3],
                                 return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([first[0], second[0]], 2), ref[0])
    assert torch.equal(torch.cat([first[1], second[1]], 3), ref[1])
    assert torch.equal(second[2], ref[2]) and torch.equal(second[3], ref[3])


def test_la_entry_state_and_empty_sequence():
    inp = _case(heads=2, seqlen=600, d_key=16)
    g = np.random.default_rng(3)
    S0 = g.standard_normal((1, 2, 16, 64)).astype(np.float32)
    dS0 = g.standard_normal((1, 1, 2, 16, 64)).astype(np.float32)
    o, do, S, dS = _run(inp, S_in=torch.from_numpy(S0), dS_in=torch.from_numpy(dS0), return_state=True)
    oo, doo, So, dSo = oracle.la_scan_jvp(*[inp[n] for n in NAMES], state=(S0, dS0))
    for got, ref in ((o, oo), (do, doo), (S, So), (dS, dSo)):
        assert gu.rel_l2(got.cpu().numpy(), ref) < gu.TOL
    d = _dev(inp)
    out = binding.la_scan_jvp(*[t[..., :0, :] for t in d], S_in=torch.from_numpy(S0), return_state=True)
    torch.cuda.synchronize()
    assert np.array_equal(out[2].cpu().numpy(), S0) and torch.all(out[3] == 0)


def test_la_zero_direction_is_exactly_zero():
    inp = _case(heads=2, seqlen=500, d_key=16)
    for n in ("dq", "dk", "dv", "dg"):
        inp[n][:] = 0.0
    _, do = _run(inp)
    assert torch.all(do == 0)


def test_la_argument_checks():
    for kw, code in ((dict(DK=48), "UNSUPPORTED"), (dict(DV=96), "UNSUPPORTED"), (dict(K=3), "UNSUPPORTED"),
                     (dict(L=-1), "INVALID_ARG")):
        a = dict(B=1, H=2, L=100, DK=16, DV=64, K=1)
        a.update(kw)
        with pytest.raises(RuntimeError, match=code):
            binding.la_plan(*a.values())
    pr = binding.make_la_params(1, 2, 100, 16, 64, 1)
    lib = binding.lib()
    assert lib.pgf_la_scan_jvp(*([None] * 8), ctypes.byref(pr), None, None, None) == -3   # no workspace
    inp = _case(heads=2, seqlen=64, d_key=16)
    d = _dev(inp)
    with pytest.raises(ValueError, match="float32"):
        binding.la_scan_jvp(*([d[0].double()] + d[1:]))
