"""The library from a plain C++ caller (tests/native/pgf_c_caller.cpp): no
Python and no torch in the process that calls it, buffers from hipMalloc,
a stream from hipStreamCreate.  The caller runs as a child process on files
this test writes; its outputs are compared with the fp64 oracle, and the
allocation-free entry point's with pgf_scan_jvp's bit for bit."""
import os
import subprocess

import numpy as np
import pytest

from oracle import oracle
from paper_2512_23068_amd import inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

CALLER = os.path.join(gu.ROOT, "tests", "native", "pgf_c_caller")


@pytest.mark.parametrize("L,N,K", [(777, 16, 2), (3000, 64, 8)])
def test_plain_c_caller(tmp_path, L, N, K):
    if not os.path.exists(CALLER):
        pytest.fail("tests/native/pgf_c_caller is not built (run __graft_entry__.build())")
    cfg = inputs.get_config("mamba130m").with_(batch=2, seqlen=L, d_inner=96, d_state=N, n_dirs=K)
    inp = inputs.make_inputs(cfg)
    with open(tmp_path / "sizes.txt", "w") as f:
        f.write(f"{cfg.batch} {L} {cfg.d_inner} {N} {K}\n")
    for name in ("x", "dx", "A", "w_delta", "b_delta", "W_B", "W_C"):
        np.ascontiguousarray(inp[name], dtype=np.float32).tofile(tmp_path / f"{name}.bin")
    print(f"case plain C caller L={L} N={N} K={K}", flush=True)
    r = subprocess.run([CALLER, str(tmp_path)], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "without workspace: PGF_ERR_WORKSPACE" in r.stdout
    y = np.fromfile(tmp_path / "y.bin", dtype=np.float32).reshape(inp["x"].shape)
    dy = np.fromfile(tmp_path / "dy.bin", dtype=np.float32).reshape(inp["dx"].shape)
    yo, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp)
    gu.assert_close(y, dy, yo, dyo, what=f"C caller L={L} N={N} K={K}")
    assert "pgf_scan_jvp_noalloc: PGF_OK" in r.stdout
    y_na = np.fromfile(tmp_path / "y_noalloc.bin", dtype=np.float32).reshape(inp["x"].shape)
    dy_na = np.fromfile(tmp_path / "dy_noalloc.bin", dtype=np.float32).reshape(inp["dx"].shape)
    assert np.array_equal(y_na, y) and np.array_equal(dy_na, dy)
