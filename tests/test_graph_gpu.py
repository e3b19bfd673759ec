"""Stream capture: a call captured into a HIP graph (through torch) and
replayed several times, with eager work and synchronisations between the
replays, gives the eager result bit for bit -- for a call of many host
blocks (whose projections run on the helper stream, forked from and joined
back to the captured stream) and for a single-block call, and for the
parameter flows (with the output map and the step size's flows), the
second-order flow and linear attention.  The library clears its state with
kernels, never with memset nodes."""
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


def _capture(fn):
    """Warm fn up on a side stream, then capture one call of it."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_graph_parameter_flows():
    """The parameter flows under capture, several host blocks: the gradients
    are added to, so each replay starts from buffers zeroed eagerly, and
    every replay equals the eager call (output map and step-size flows on)."""
    import numpy as np
    from paper_2512_23068_amd import inputs
    inp = gu.custom("mamba130m", batch=1, seqlen=1500, d_inner=256)
    inp["gy"] = inputs.make_adjoint(inp["cfg"])
    inp["D_res"] = np.random.default_rng(3).standard_normal(256).astype(np.float32)
    x, _ = gu.inputs_to_dev(inp)
    gy = torch.from_numpy(inp["gy"]).to(gu.dev())
    prm = gu.params_to_dev(inp)
    kw = dict(seg_len=64, chunk_segs=2, act="silu", delta_params=True)
    info = binding.plan(1, 1500, 256, 16, 1, order=3, seg_len=64, chunk_segs=2, act="silu", delta_flows=True)
    assert info["n_chunks"] > 1
    ref = binding.param_grads(x, gy, prm, **kw)
    torch.cuda.synchronize()
    y = torch.empty_like(ref[0])
    grads = tuple(torch.zeros_like(r) for r in ref[1:])
    ws = torch.empty(info["workspace_bytes"], device=gu.dev(), dtype=torch.uint8)
    g = _capture(lambda: binding.param_grads(x, gy, prm, grads=grads, out=y, workspace=ws, **kw))
    for rep in range(3):
        y.fill_(7.0)
        for t in grads:
            t.zero_()
        ws.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref[0]) and all(torch.equal(a, b) for a, b in zip(grads, ref[1:])), rep


def test_graph_second_order_and_linear_attention():
    import numpy as np
    from paper_2512_23068_amd import inputs
    inp = gu.custom("mamba130m", batch=1, seqlen=1200, d_inner=128, n_dirs=2)
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    ref = binding.scan_jvp2(x, dx, prm, seg_len=64, chunk_segs=3)
    torch.cuda.synchronize()
    outs = tuple(torch.empty_like(r) for r in ref)
    ws = torch.empty(binding.workspace_bytes(1, 1200, 128, 16, 2, seg_len=64, chunk_segs=3, order=2),
                     device=gu.dev(), dtype=torch.uint8)
    g = _capture(lambda: binding.scan_jvp2(x, dx, prm, seg_len=64, chunk_segs=3, out=outs, workspace=ws))
    for rep in range(2):
        for t in outs:
            t.fill_(3.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip(outs, ref)), ("order 2", rep)

    cfg = inputs.LA_BY_NAME["la_tiny"].with_(heads=2, seqlen=1100, d_key=32)
    la = inputs.make_la_inputs(cfg)
    d = [torch.from_numpy(np.ascontiguousarray(la[n])).to(gu.dev()) for n in ("q", "k", "v", "g", "dq", "dk", "dv",
                                                                               "dg")]
    ref = binding.la_scan_jvp(*d, seg_len=64, chunk_segs=3)
    torch.cuda.synchronize()
    outs = tuple(torch.empty_like(r) for r in ref)
    ws = torch.empty(binding.la_plan(1, 2, 1100, 32, cfg.d_value, 1, seg_len=64, chunk_segs=3)["workspace_bytes"],
                     device=gu.dev(), dtype=torch.uint8)
    g = _capture(lambda: binding.la_scan_jvp(*d, seg_len=64, chunk_segs=3, out=outs, workspace=ws))
    for rep in range(2):
        for t in outs:
            t.fill_(-3.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip(outs, ref)), ("linear attention", rep)
