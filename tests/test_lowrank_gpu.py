"""The low-rank step size (Mamba's step-size projection through a rank-R
bottleneck) on the GPU against the fp64 oracle; the rank-D identity
projection equals the per-channel step size to rounding; block-size
invariance; argument limits."""
import numpy as np
import pytest
import torch

from oracle import oracle
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _low_rank(inp, R, seed=13):
    D = inp["A"].shape[0]
    r = np.random.default_rng(seed)
    inp["W_dx"] = (r.standard_normal((D, R)) / np.sqrt(D)).astype(np.float32)
    inp["W_dt"] = (r.uniform(-1.0, 1.0, (R, D)) / np.sqrt(R)).astype(np.float32)
    return inp


_run = gu.run


def _check(inp, what, **kw):
    print(f"case {what}", flush=True)
    y, dy = _run(inp, **kw)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, act=kw.get("act", "identity"))
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what=what)


@pytest.mark.parametrize("R,N,K,seg", [(48, 16, 1, 0), (16, 16, 2, 0), (5, 8, 1, -1), (128, 4, 2, 64),
                                       (100, 16, 1, 128)])
def test_low_rank_parity(R, N, K, seg):
    # 1100 steps: several projection tiles and a ragged tail; D = 320 is not a
    # multiple of the 128-channel z tile
    inp = _low_rank(gu.custom("mamba130m", batch=2, seqlen=1100, d_inner=320, d_state=N, n_dirs=K), R)
    _check(inp, f"low rank R={R} N={N} K={K} seg={seg}", seg_len=seg)


def test_low_rank_with_output_map_and_bf16():
    inp = _low_rank(gu.custom("mamba130m", batch=1, seqlen=900, d_inner=384, n_dirs=1), 24)
    inp["D_res"] = np.random.default_rng(2).standard_normal(384).astype(np.float32)
    _check(inp, "low rank + silu + D_res", act="silu")
    _check(_low_rank(gu.custom("stiff128k", seqlen=1200, d_inner=256), 32), "low rank stiff bf16")


def test_identity_projection_matches_depthwise():
    """R = D, W_dx = I, W_dt = diag(w): z = x*w + b, the per-channel step
    size; the two paths round differently (the products on the matrix cores
    add exact zeros), so they agree to rounding, not bit for bit."""
    inp = gu.custom("mamba130m", batch=1, seqlen=600, d_inner=128, n_dirs=2)
    y1, dy1 = _run(inp)
    lr = dict(inp, W_dx=np.eye(128, dtype=np.float32), W_dt=np.diag(inp["w_delta"]).astype(np.float32))
    y2, dy2 = _run(lr)
    assert gu.rel_l2(y2.cpu().numpy(), y1.cpu().numpy()) < 1e-6
    assert gu.rel_l2(dy2.cpu().numpy(), dy1.cpu().numpy()) < 1e-6


def test_low_rank_block_invariance():
    inp = _low_rank(gu.custom("mamba130m", batch=2, seqlen=1000, d_inner=128, n_dirs=2), 16)
    ref = _run(inp, seg_len=64, chunk_segs=1, return_state=True)
    for cs in (3, 0):
        got = _run(inp, seg_len=64, chunk_segs=cs, return_state=True)
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs


def test_low_rank_limits():
    inp = _low_rank(gu.custom("tiny", seqlen=64, d_inner=128), 129)
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        _run(inp)
    inp = _low_rank(gu.custom("tiny", seqlen=64, d_inner=128), 8)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        _run(inp, drive="zoh")
    inp = _low_rank(gu.custom("tiny", seqlen=64, d_inner=128, n_dirs=4), 8)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        _run(inp)
