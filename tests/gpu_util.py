"""Helpers of the GPU tests: run the HIP path on seeded inputs and compare
with the fp64 oracle."""
import json
import os

import numpy as np
import torch

from oracle import oracle
from paper_2512_23068_amd import binding, inputs

PARAM_KEYS = ("A", "w_delta", "b_delta", "W_B", "W_C", "b_B", "b_C", "D_res", "A_im", "W_dx", "W_dt")
INT_KEYS = ("n_groups",)
TOL = 1e-5   # relative L2, f32 state against the fp64 oracle
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# Where the full-size parity tests record their errors (one JSON object,
# merged key by key; the summary under profiles/ is copied from it).
PARITY_JSON = os.environ.get("PGF_PARITY_JSON", os.path.join(ROOT, "gpurun_out", "parity_full.json"))


def dev():
    return torch.device("cuda:0")


def params_to_dev(inp):
    out = {k: torch.from_numpy(np.ascontiguousarray(inp[k])).to(dev()) for k in PARAM_KEYS if k in inp}
    out.update({k: inp[k] for k in INT_KEYS if k in inp})
    return out


def inputs_to_dev(inp, bf16=None):
    if bf16 is None:
        bf16 = inp.get("cfg") is not None and inp["cfg"].in_dtype == "bf16"
    x = torch.from_numpy(inp["x"]).to(dev())
    dx = torch.from_numpy(inp["dx"]).to(dev())
    if bf16:   # the values are already bf16-representable: the cast is exact
        x, dx = x.to(torch.bfloat16), dx.to(torch.bfloat16)
    return x, dx


def run(inp, bf16=None, **kw):
    x, dx = inputs_to_dev(inp, bf16)
    out = binding.scan_jvp(x, dx, params_to_dev(inp), **kw)
    torch.cuda.synchronize()
    return out


def rel_l2(got, ref):
    """||got - ref|| / ||ref|| in fp64; complex inputs compare both the real
    and the imaginary parts."""
    cplx = np.iscomplexobj(got) or np.iscomplexobj(ref)
    dt = np.complex128 if cplx else np.float64
    got = np.asarray(got, dtype=dt)
    ref = np.asarray(ref, dtype=dt)
    den = np.linalg.norm(ref.ravel())
    return float(np.linalg.norm((got - ref).ravel()) / (den if den > 0 else 1.0))


def sum_error(got, ref, scale):
    """||got - ref|| / ||scale|| in fp64, for accumulated sums whose terms
    take both signs: scale holds, per output, the sum of the absolute values
    of its terms (the condition of the summation), so that the measure does
    not grow where the terms cancel."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(np.asarray(scale, dtype=np.float64).ravel())
    return float(np.linalg.norm((got - ref).ravel()) / (den if den > 0 else 1.0))


def assert_close(y, dy, yo, dyo, tol=TOL, what=""):
    ey = rel_l2(y, yo)
    edys = [rel_l2(dy[k], dyo[k]) for k in range(dyo.shape[0])]
    print(f"{what} rel_l2 y={ey:.3e} dy={max(edys):.3e}", flush=True)
    assert np.all(np.isfinite(y)) and np.all(np.isfinite(dy))
    assert ey <= tol, (what, ey)
    assert max(edys) <= tol, (what, edys)
    return ey, max(edys)


def custom(name, **kw):
    """A workload with the recipe of `name` and some sizes changed."""
    return inputs.make_inputs(inputs.get_config(name).with_(**kw))


def record(key, values):
    """Merges {key: values} into the parity record (PARITY_JSON)."""
    os.makedirs(os.path.dirname(PARITY_JSON), exist_ok=True)
    data = {}
    if os.path.exists(PARITY_JSON):
        with open(PARITY_JSON) as f:
            data = json.load(f)
    data[key] = values
    with open(PARITY_JSON + ".tmp", "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
    os.replace(PARITY_JSON + ".tmp", PARITY_JSON)
