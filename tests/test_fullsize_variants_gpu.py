"""The benchmarked configurations of the follow-on paths at pulse128k's full
sizes (B=1, L=131072, D=1536, N=16), in the default plan the benchmark
times, against the fp64 oracle over the whole sequence on one seeded
channel of every 64-channel block (every workgroup's block of channels)
and the first and last channel: the second-order flow (two N(0,1)
directions), the zero-order-hold drive, SiLU with a residual weight, the
complex S4D-Lin spectrum, four channel groups and the rank-48 step-size
projection.  The parameter recipes are the ones bench.py uses
(inputs.variant_params); the errors go to the parity record."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _channels(D, block=64, seed=1):
    g = np.random.default_rng(seed)
    picks = [int(g.integers(s, min(s + block, D))) for s in range(0, D, block)]
    return np.unique(np.concatenate([[0, D - 1], picks])).astype(np.int64)


def _record(key, sel, errs):
    gu.record(key, {"channels_compared": int(len(sel)), **{k: float(v) for k, v in errs.items()}})


def _sampled(y, dy, sel):
    idx = torch.from_numpy(sel).to(gu.dev())
    return y.index_select(-1, idx).cpu().numpy(), dy.index_select(-1, idx).cpu().numpy()


VARIANTS = {
    "zoh": (dict(), dict(drive="zoh")),
    "silu_dres": (dict(dres=True), dict(act="silu")),
    "s4dlin": (dict(complex_a=True), dict()),
    "s4dlin_silu_dres": (dict(complex_a=True, dres=True), dict(act="silu")),
    "s4dlin_zoh": (dict(complex_a=True), dict(drive="zoh")),
    "groups4": (dict(groups=4), dict()),
    "lowrank48": (dict(lowrank=48), dict()),
}


@pytest.mark.parametrize("name", sorted(VARIANTS))
def test_variant_full_size_sampled_channels(name):
    pkw, rkw = VARIANTS[name]
    cfg = inputs.get_config("pulse128k")
    print(f"case pulse128k-{name}: inputs", flush=True)
    inp = inputs.make_inputs(cfg)
    prm = inputs.variant_params({k: inp[k] for k in ("A", "w_delta", "b_delta", "W_B", "W_C")}, cfg, **pkw)
    x, dx = gu.inputs_to_dev(inp)
    print(f"case pulse128k-{name}: GPU scan", flush=True)
    y, dy = binding.scan_jvp(x, dx, gu.params_to_dev(prm), **rkw)
    torch.cuda.synchronize()
    sel = _channels(cfg.d_inner)
    yg, dyg = _sampled(y, dy, sel)
    del x, dx, y, dy
    torch.cuda.empty_cache()
    print(f"case pulse128k-{name}: oracle on channels {sel.tolist()}", flush=True)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], prm, channels=sel, chunk=4096, **rkw)
    _record(f"pulse128k_{name}", sel, {"y_rel_l2": gu.rel_l2(yg, yo), "dy_rel_l2": gu.rel_l2(dyg, dyo)})
    gu.assert_close(yg, dyg, yo, dyo, what=f"pulse128k-{name}")


def test_second_order_full_size_sampled_channels():
    cfg = inputs.get_config("pulse128k").with_(n_dirs=2, dx_kind="normal")
    print("case pulse128k-order2: inputs", flush=True)
    inp = inputs.make_inputs(cfg)
    x, dx = gu.inputs_to_dev(inp)
    print("case pulse128k-order2: GPU scan", flush=True)
    y, dy, d2y = binding.scan_jvp2(x, dx, gu.params_to_dev(inp))
    torch.cuda.synchronize()
    sel = _channels(cfg.d_inner)
    yg, dyg = _sampled(y, dy, sel)
    d2yg = d2y.index_select(-1, torch.from_numpy(sel).to(gu.dev())).cpu().numpy()
    del x, dx, y, dy, d2y
    torch.cuda.empty_cache()
    print(f"case pulse128k-order2: oracle on channels {sel.tolist()}", flush=True)
    (yo, yvo, ywo, yvwo), _ = oracle.scan_jvp2(inp["x"], inp["dx"][0], inp["dx"][1], inp, channels=sel, chunk=4096)
    e = gu.rel_l2(d2yg, yvwo)
    print(f"pulse128k-order2 rel_l2 d2y={e:.3e}", flush=True)
    _record("pulse128k_order2", sel, {"y_rel_l2": gu.rel_l2(yg, yo), "dy_v_rel_l2": gu.rel_l2(dyg[0], yvo),
                                      "dy_w_rel_l2": gu.rel_l2(dyg[1], ywo), "d2y_rel_l2": e})
    gu.assert_close(yg, dyg, yo, np.stack([yvo, ywo]), what="pulse128k-order2")
    assert np.all(np.isfinite(d2yg)) and e <= gu.TOL, e
