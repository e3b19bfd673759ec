"""Second-order (App. G Hessian flow) HIP path against the fp64 oracle and
against the first-order path: parity of y, both first-order flows and the
mixed flow; bit-identical y and dy to pgf_scan_jvp on the same directions;
block-size invariance, split-call hand-off of all four states, exact zeros
ahead of the directions, and argument checks."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _run2(inp, **kw):
    x, dx = gu.inputs_to_dev(inp)
    out = binding.scan_jvp2(x, dx, gu.params_to_dev(inp), **kw)
    torch.cuda.synchronize()
    return out


def _check2(inp, what, **kw):
    print(f"case {what}", flush=True)
    y, dy, d2y = _run2(inp, **kw)
    (yo, yvo, ywo, yvwo), _ = oracle.scan_jvp2(inp["x"], inp["dx"][0], inp["dx"][1], inp)
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, np.stack([yvo, ywo]), what=what)
    e = gu.rel_l2(d2y.cpu().numpy(), yvwo)
    print(f"{what} rel_l2 d2y={e:.3e}", flush=True)
    assert np.all(np.isfinite(d2y.cpu().numpy())) and e <= gu.TOL, (what, e)


@pytest.mark.parametrize("N,seg", [(16, 0), (8, 0), (4, 0), (16, -1), (16, 64), (32, 0), (64, 64), (32, -1)])
def test_second_order_parity(N, seg):
    inp = gu.custom("mamba130m", batch=2, seqlen=1100, d_inner=70, d_state=N, n_dirs=2)
    _check2(inp, f"order2 N={N} seg={seg}", seg_len=seg)


def test_second_order_bf16_stiff():
    inp = gu.custom("stiff128k", seqlen=1500, d_inner=64, n_dirs=2)
    _check2(inp, "order2 stiff bf16")


def test_first_order_outputs_match_pgf_scan_jvp():
    inp = gu.custom("mamba130m", batch=1, seqlen=900, d_inner=96, n_dirs=2)
    for seg in (128, -1):
        y2, dy2, _ = _run2(inp, seg_len=seg, chunk_segs=4)
        y1, dy1 = gu.run(inp, seg_len=seg, chunk_segs=4)
        assert torch.equal(y1, y2) and torch.equal(dy1, dy2), seg


def test_second_order_block_invariance_and_handoff():
    inp = gu.custom("mamba130m", batch=2, seqlen=1000, d_inner=48, n_dirs=2)
    ref = _run2(inp, seg_len=64, chunk_segs=1, return_state=True)
    for cs in (3, 0):
        got = _run2(inp, seg_len=64, chunk_segs=cs, return_state=True)
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    s = 384
    a = binding.scan_jvp2(x[:, :s], dx[:, :, :s], prm, seg_len=64, return_state=True)
    b = binding.scan_jvp2(x[:, s:], dx[:, :, s:], prm, seg_len=64, h_in=a[3], dh_in=a[4], d2h_in=a[5],
                          return_state=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a[0], b[0]], 1), ref[0])
    assert torch.equal(torch.cat([a[1], b[1]], 2), ref[1])
    assert torch.equal(torch.cat([a[2], b[2]], 1), ref[2])
    for i in (3, 4, 5):
        assert torch.equal(b[i], ref[i]), i


def test_second_order_entry_state_matches_oracle():
    inp = gu.custom("mamba130m", batch=1, seqlen=700, d_inner=40, n_dirs=2)
    g = np.random.default_rng(41)
    st = [g.standard_normal((1, 40, 16)).astype(np.float32) for _ in range(4)]
    y, dy, d2y, h, dh, d2h = _run2(inp, h_in=torch.from_numpy(st[0]),
                                   dh_in=torch.from_numpy(np.stack([st[1], st[2]])),
                                   d2h_in=torch.from_numpy(st[3]), return_state=True)
    (yo, yvo, ywo, yvwo), so = oracle.scan_jvp2(inp["x"], inp["dx"][0], inp["dx"][1], inp, state=tuple(st))
    assert gu.rel_l2(d2y.cpu().numpy(), yvwo) < gu.TOL
    assert gu.rel_l2(d2h.cpu().numpy(), so[3]) < gu.TOL and gu.rel_l2(dh[1].cpu().numpy(), so[2]) < gu.TOL


def test_second_order_zero_ahead_of_directions():
    inp = gu.custom("mamba130m", batch=1, seqlen=800, d_inner=32, n_dirs=2)
    t0 = 333
    inp["dx"][0, :, :t0] = 0.0
    y, dy, d2y = _run2(inp)
    assert torch.all(d2y[:, :t0] == 0) and torch.all(dy[0, :, :t0] == 0)
    assert torch.all(d2y[:, t0:].abs().sum(-1) > 0)


def test_second_order_argument_checks():
    inp = gu.custom("tiny", seqlen=64, n_dirs=2)
    with pytest.raises(ValueError, match="two directions"):
        x, dx = gu.inputs_to_dev(inp)
        binding.scan_jvp2(x, dx[:1], gu.params_to_dev(inp))
    # order 2 takes no variant; order mismatches are refused
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        binding.plan(1, 64, 16, 32, 2, order=2, drive="zoh")
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        binding.plan(1, 64, 16, 16, 1, order=2)
    pr = binding.make_params(1, 64, 16, 16, 2, order=1)
    lib = binding.lib()
    rc = lib.pgf_scan_jvp2(None, None, ctypes.byref(pr), None, None, None, None)
    assert rc == -1
