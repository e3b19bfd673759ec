"""The largest host block the planner accepts, on the GPU.

The kernels address one host block with 32-bit element offsets t*D + d, and
the planner admits blocks of up to 2^30 elements.  With D = 16384 channels
a block of 65536 steps is exactly that bound, in the sequential evaluation
(16 units of 4096 steps) and in the segmented one (256 segments of 256
steps); the call below runs two such plans over 65536 + 300 steps (a full
block, then a ragged one) and compares sampled channels, the first and the
last among them, over the whole sequence with the fp64 oracle.  One more
unit or segment per block is rejected before anything is launched."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

D = 16384
BLOCK = 65536                      # steps per host block at the bound
L = BLOCK + 300
PLANS = ((-1, BLOCK // 4096), (256, BLOCK // 256))   # (seg_len, chunk_segs)


def test_largest_host_block():
    for seg, cs in PLANS:
        p = binding.plan(1, L, D, 16, 1, seg_len=seg, chunk_segs=cs)
        assert p["chunk_len"] * D == 2 ** 30 and p["n_chunks"] == 2, p
        with pytest.raises(RuntimeError, match="INVALID_ARG"):
            binding.plan(1, L, D, 16, 1, seg_len=seg, chunk_segs=cs + 1)
    print(f"case max host block D={D} L={L}", flush=True)
    inp = gu.custom("mamba130m", batch=1, seqlen=L, d_inner=D, dx_kind="normal")
    g = np.random.default_rng(31)
    ch = np.unique(np.concatenate([[0, D - 1], g.choice(np.arange(1, D - 1), 6, replace=False)]))
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, channels=ch, chunk=8192)
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    idx = torch.from_numpy(ch).to(gu.dev())
    for seg, cs in PLANS:
        y, dy = binding.scan_jvp(x, dx, prm, seg_len=seg, chunk_segs=cs)
        torch.cuda.synchronize()
        gu.assert_close(y.index_select(-1, idx).cpu().numpy(), dy.index_select(-1, idx).cpu().numpy(), yo, dyo,
                        what=f"max block seg={seg} chunk_segs={cs}")
        del y, dy
    del x, dx, prm
    torch.cuda.empty_cache()
