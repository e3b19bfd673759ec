"""Stream capture: a call captured into a HIP graph (through torch) and
replayed several times, with eager work and synchronisations between the
replays, gives the eager result bit for bit -- for a call of many host
blocks (whose projections run on the helper stream, forked from and joined
back to the captured stream) and for a single-block call.  The library
clears its state with kernels, never with memset nodes."""
import pytest
import torch

from paper_2512_23068_amd import binding
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("chunk_segs", [2, 0])
def test_graph_replays_equal_eager(chunk_segs):
    inp = gu.custom("mamba130m", batch=1, seqlen=1500, d_inner=256, n_dirs=1)
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    kw = dict(seg_len=64, chunk_segs=chunk_segs)
    info = binding.plan(1, 1500, 256, 16, 1, **kw)
    print(f"case graph chunk_segs={chunk_segs}: {info['n_chunks']} host blocks", flush=True)
    assert (info["n_chunks"] > 1) == (chunk_segs == 2)
    y0, dy0 = binding.scan_jvp(x, dx, prm, **kw)   # eager reference; creates the helper stream
    torch.cuda.synchronize()
    y, dy = torch.empty_like(y0), torch.empty_like(dy0)
    ws = torch.empty(info["workspace_bytes"], device=gu.dev(), dtype=torch.uint8)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                  # warm-up outside the capture
        binding.scan_jvp(x, dx, prm, out=(y, dy), workspace=ws, **kw)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        binding.scan_jvp(x, dx, prm, out=(y, dy), workspace=ws, **kw)
    torch.cuda.synchronize()
    for rep in range(3):
        y.fill_(7.0)                               # eager work between replays
        dy.fill_(-7.0)
        ws.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y0) and torch.equal(dy, dy0), rep
