"""Channel groups with their own B and C (Mamba-style grouped projections)
on the GPU against the fp64 oracle; groups that share their weights equal
one group bit for bit; block-size invariance; argument limits."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _grouped(inp, G, seed=11):
    D, N = inp["A"].shape
    r = np.random.default_rng(seed)
    inp["n_groups"] = G
    inp["W_B"] = (r.standard_normal((D, G * N)) / np.sqrt(D)).astype(np.float32)
    inp["W_C"] = (r.standard_normal((D, G * N)) / np.sqrt(D)).astype(np.float32)
    inp["b_B"] = r.standard_normal(G * N).astype(np.float32)
    inp["b_C"] = r.standard_normal(G * N).astype(np.float32)
    return inp


def _check(inp, what, **kw):
    print(f"case {what}", flush=True)
    y, dy = gu.run(inp, **kw)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, act=kw.get("act", "identity"))
    gu.assert_close(y.cpu().numpy(), dy.cpu().numpy(), yo, dyo, what=what)


@pytest.mark.parametrize("G,N,K,seg", [(2, 16, 1, 0), (4, 16, 2, 0), (2, 8, 1, -1), (4, 4, 1, 64)])
def test_groups_parity(G, N, K, seg):
    inp = _grouped(gu.custom("mamba130m", batch=2, seqlen=1100, d_inner=256, d_state=N, n_dirs=K), G)
    _check(inp, f"groups G={G} N={N} K={K} seg={seg}", seg_len=seg)


def test_groups_with_output_map_and_bf16():
    inp = _grouped(gu.custom("mamba130m", batch=1, seqlen=900, d_inner=384, n_dirs=1), 2)
    inp["D_res"] = np.random.default_rng(2).standard_normal(384).astype(np.float32)
    _check(inp, "groups + silu + D_res", act="silu")
    _check(_grouped(gu.custom("stiff128k", seqlen=1200, d_inner=256), 2), "groups stiff bf16")


def test_shared_group_weights_equal_one_group():
    """Four groups with the same weights give one group's result.  The
    grouped projection has 128 columns, which run on the split-plane bf16
    matrix-core form, one group's 32 on the f32 matrix cores: both round
    like f32 products, so the outputs agree to f32 rounding; two groups (64
    columns) against four (128) take the same form and agree bit for bit."""
    inp = gu.custom("mamba130m", batch=2, seqlen=700, d_inner=256, n_dirs=2)
    y1, dy1 = gu.run(inp)

    def tiled(G):
        return dict(inp, n_groups=G, W_B=np.tile(inp["W_B"], (1, G)), W_C=np.tile(inp["W_C"], (1, G)),
                    b_B=np.zeros(G * 16, np.float32), b_C=np.zeros(G * 16, np.float32))

    y4, dy4 = gu.run(tiled(4))
    ey = gu.rel_l2(y4.cpu().numpy(), y1.cpu().numpy())
    edy = gu.rel_l2(dy4.cpu().numpy(), dy1.cpu().numpy())
    print(f"4 shared groups vs one group: y {ey:.2e} dy {edy:.2e}", flush=True)
    assert ey < 1e-6 and edy < 1e-6
    y2, dy2 = gu.run(tiled(2))
    assert torch.equal(y2, y4) and torch.equal(dy2, dy4)


def test_groups_block_invariance():
    inp = _grouped(gu.custom("mamba130m", batch=2, seqlen=1000, d_inner=128, n_dirs=2), 2)
    ref = gu.run(inp, seg_len=64, chunk_segs=1, return_state=True)
    for cs in (3, 0):
        got = gu.run(inp, seg_len=64, chunk_segs=cs, return_state=True)
        for a, b in zip(got, ref):
            assert torch.equal(a, b), cs


def test_group_limits():
    inp = _grouped(gu.custom("tiny", seqlen=64, d_inner=96), 2)      # 48 channels per group
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        gu.run(inp)
    inp = _grouped(gu.custom("tiny", seqlen=64, d_inner=128), 2)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        gu.run(inp, drive="zoh")
    inp = _grouped(gu.custom("tiny", seqlen=64, d_inner=128, n_dirs=4), 2)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        gu.run(inp)
    inp = _grouped(gu.custom("tiny", seqlen=64, d_inner=192), 3)      # G*N = 48: not a power of two
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        gu.run(inp)
