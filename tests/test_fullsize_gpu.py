"""The five benchmark workloads at their full sizes, in the launch
configuration the benchmark times (the default plan), against the fp64
oracle on sampled channels over the whole sequence (the oracle computes any
channel on its own; the projections still contract over every channel).
Also: peak device memory minus the IO payload is the same for every L."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

# channels compared per workload: first, last, and a seeded spread
def _channels(D, n=6, seed=0):
    g = np.random.default_rng(seed)
    extra = g.choice(np.arange(1, D - 1), size=min(n, max(D - 2, 0)), replace=False)
    return np.unique(np.concatenate([[0, D - 1], extra])).astype(np.int64)


def _run_full(name, n_ch=6):
    cfg = inputs.get_config(name)
    print(f"case {name}: generating inputs", flush=True)
    inp = inputs.make_inputs(cfg)
    sel = _channels(cfg.d_inner, n_ch)
    x, dx = gu.inputs_to_dev(inp)
    print(f"case {name}: GPU scan", flush=True)
    y, dy = binding.scan_jvp(x, dx, gu.params_to_dev(inp))
    torch.cuda.synchronize()
    idx = torch.from_numpy(sel).to(gu.dev())
    yg = y.index_select(-1, idx).cpu().numpy()
    dyg = dy.index_select(-1, idx).cpu().numpy()
    del x, dx, y, dy
    torch.cuda.empty_cache()
    print(f"case {name}: oracle on channels {sel.tolist()}", flush=True)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, channels=sel, chunk=4096)
    return cfg, yg, dyg, yo, dyo


@pytest.mark.parametrize("name", ["mamba130m", "pulse128k", "stiff128k", "multidir"])
def test_full_workload_sampled_channels(name):
    cfg, yg, dyg, yo, dyo = _run_full(name, n_ch=6 if name != "multidir" else 3)
    gu.assert_close(yg, dyg, yo, dyo, what=name)
    if name == "pulse128k":
        # the impulse response's tail over the last 1024 steps, reported
        tail = gu.rel_l2(dyg[:, :, -1024:], dyo[:, :, -1024:])
        mag = float(np.abs(dyo[:, :, -1024:]).max())
        print(f"pulse128k tail rel_l2(dy, last 1024 steps) = {tail:.3e} (max |dy| there {mag:.3e})", flush=True)
        assert np.isfinite(tail) and mag > 0


def test_peak_memory_flat_in_L():
    """Peak allocated bytes minus the IO payload (x, dx, y, dy) do not depend
    on L (Sec. 4.3: only the O(1) tile is differentiation overhead)."""
    cfg = inputs.get_config("pulse128k")
    D, N = cfg.d_inner, cfg.d_state
    prm = gu.params_to_dev(inputs.make_params(cfg))
    incr = []
    for L in (8192, 16384, 32768, 65536, 131072):
        torch.cuda.empty_cache()
        x = torch.randn(1, L, D, device=gu.dev(), dtype=torch.float32)
        dx = torch.randn(1, 1, L, D, device=gu.dev(), dtype=torch.float32)
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        y, dy = binding.scan_jvp(x, dx, prm)
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated()
        outs = y.numel() * 4 + dy.numel() * 4
        incr.append(peak - base - outs)
        print(f"L={L}: peak-minus-payload increment {incr[-1]} bytes", flush=True)
        del x, dx, y, dy
    assert len(set(incr)) == 1, incr
    assert incr[0] <= binding.workspace_bytes(1, 131072, D, N, 1) + (1 << 20)
