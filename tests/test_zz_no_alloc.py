"""pgf_scan_jvp_noalloc (the entry point for callers that cannot allocate)
against pgf_scan_jvp through the C ABI: bit-identical outputs on two calls
in a row (the second smaller, so the shared static scratch still holds the
first call's data), a call whose plan is cut to fit the scratch, no device
memory taken by the calls, and the rejection of a call that cannot fit."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2512_23068_amd import binding
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _both(inp, **kw):
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    ref = binding.scan_jvp(x, dx, prm, **kw)
    out = (torch.full_like(ref[0], np.nan), torch.full_like(ref[1], np.nan))
    torch.cuda.synchronize()
    got = binding.scan_jvp_noalloc(x, dx, prm, out, **kw)
    torch.cuda.synchronize()
    return ref, got


def _assert_equal(ref, got, what):
    for a, b in zip(ref, got):
        assert torch.equal(a, b), what


def test_noalloc_two_calls_match_scan_jvp():
    # first a larger call (1536 channels, 8 host blocks of 2048 steps), then a
    # smaller one with two directions: the second must read nothing of what
    # the first left in the scratch
    big = gu.custom("mamba130m", seqlen=16000, d_inner=1536)
    ref, got = _both(big, chunk_segs=8)
    print("noalloc call 1: equal", flush=True)
    _assert_equal(ref, got, "call 1")
    small = gu.custom("mamba130m", batch=2, seqlen=1500, d_inner=200, n_dirs=2)
    ref, got = _both(small)
    print("noalloc call 2: equal", flush=True)
    _assert_equal(ref, got, "call 2")
    # the oracle bar as well (the equality above makes it the same test)
    yo_err = gu.rel_l2(got[0].cpu().numpy(), ref[0].cpu().numpy())
    assert yo_err == 0.0


def test_noalloc_sequential_and_bf16():
    inp = gu.custom("stiff128k", seqlen=9000, d_inner=128)
    ref, got = _both(inp, seg_len=-1)
    _assert_equal(ref, got, "sequential bf16")


def test_noalloc_plan_cut_to_the_scratch():
    """D = 4096, N = 64, K = 2 with 1024-step segments: the default plan's
    workspace (365 MiB, one host block) does not fit the scratch, so the
    no-alloc call runs shorter host blocks; the outputs still equal
    pgf_scan_jvp's bit for bit."""
    B, L, D, N, K = 1, 40000, 4096, 64, 2
    assert binding.workspace_bytes(B, L, D, N, K, seg_len=1024) > (256 << 20)
    assert binding.plan(B, L, D, N, K, seg_len=1024)["n_chunks"] == 1
    inp = gu.custom("multidir", batch=B, seqlen=L, d_inner=D, d_state=N, n_dirs=K)
    ref, got = _both(inp, seg_len=1024)
    _assert_equal(ref, got, "cut plan")


def test_noalloc_allocates_nothing():
    inp = gu.custom("mamba130m", seqlen=3000, d_inner=512)
    x, dx = gu.inputs_to_dev(inp)
    prm = gu.params_to_dev(inp)
    out = (torch.empty(x.shape, device=x.device), torch.empty(dx.shape, device=x.device))
    binding.scan_jvp_noalloc(x, dx, prm, out)      # first call on the device: the array's address
    torch.cuda.synchronize()
    torch_before = torch.cuda.memory_allocated()
    free_before, _ = torch.cuda.mem_get_info()
    for _ in range(3):
        binding.scan_jvp_noalloc(x, dx, prm, out)
    torch.cuda.synchronize()
    free_after, _ = torch.cuda.mem_get_info()
    assert torch.cuda.memory_allocated() == torch_before
    assert free_after == free_before, (free_before, free_after)


def test_noalloc_rejects_a_call_beyond_the_scratch():
    # the carried state alone, (1+K)*B*N*D*4 bytes = 1.2 GB, exceeds it
    B, D, N, K = 64, 8192, 64, 8
    x = torch.zeros((B, 1, D), device=gu.dev())
    dx = torch.zeros((K, B, 1, D), device=gu.dev())
    prm = {"A": torch.full((D, N), -1.0, device=gu.dev()), "w_delta": torch.zeros(D, device=gu.dev()),
           "b_delta": torch.zeros(D, device=gu.dev()), "W_B": torch.zeros((D, N), device=gu.dev()),
           "W_C": torch.zeros((D, N), device=gu.dev())}
    y = torch.full((B, 1, D), 7.0, device=gu.dev())
    dy = torch.full((K, B, 1, D), 7.0, device=gu.dev())
    with pytest.raises(RuntimeError, match="SCRATCH"):
        binding.scan_jvp_noalloc(x, dx, prm, (y, dy))
    torch.cuda.synchronize()
    assert torch.all(y == 7.0) and torch.all(dy == 7.0)   # nothing launched
    pr = binding.make_params(B, 1, D, N, K)
    assert binding.lib().pgf_scan_jvp_noalloc(None, None, ctypes.byref(pr), None, None, None) == -1
