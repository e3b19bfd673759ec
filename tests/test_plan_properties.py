"""Property tests of the host planner through the C ABI (no GPU needed):
over random sizes and tiling overrides a plan is either refused with a
status (INVALID_ARG or UNSUPPORTED) before anything else happens, or it
covers the sequence with whole host blocks whose element offsets fit the
kernels' 32-bit addressing, its workspace does not depend on L, and the
plan and workspace entry points agree."""
import pytest
from hypothesis import given, settings, strategies as st

from paper_2512_23068_amd import binding

SEGS = [0, -1, 16, 32, 64, 128, 256, 512, 1024, 4096]


def _plan(*a, **kw):
    try:
        return binding.plan(*a, **kw)
    except RuntimeError as e:
        msg = str(e)
        assert "INVALID_ARG" in msg or "UNSUPPORTED" in msg, msg
        return None


@settings(max_examples=400, deadline=None)
@given(B=st.integers(1, 8), L=st.integers(0, 1 << 20), D=st.integers(1, 8192),
       N=st.sampled_from([4, 8, 16, 32, 64]), K=st.sampled_from([1, 2, 4, 8]),
       seg=st.sampled_from(SEGS), cs=st.integers(0, 64), bf16=st.booleans(), order=st.sampled_from([1, 2, 3]))
def test_scan_plans(B, L, D, N, K, seg, cs, bf16, order):
    if order == 2:
        K = 2
    if order == 3:
        K = 1
    dt = "bf16" if bf16 else "f32"
    kw = dict(in_dtype=dt, seg_len=seg, chunk_segs=cs, order=order)
    p = _plan(B, L, D, N, K, **kw)
    ws = binding.workspace_bytes(B, L, D, N, K, **kw)
    if p is None:
        assert ws == 0
        return
    assert ws == p["workspace_bytes"] > 0
    assert p["n_per_thread"] * p["n_split"] == N
    assert p["chunk_len"] > 0 and p["chunk_len"] * D <= 1 << 30
    assert p["n_chunks"] == -(-L // p["chunk_len"])
    if p["seg_len"] > 0:
        assert p["chunk_len"] == p["seg_len"] * p["chunk_segs"]
        if seg > 0:
            assert p["seg_len"] == seg
        if cs > 0:
            assert p["chunk_segs"] == cs
    else:
        assert p["chunk_len"] % 4096 == 0
    # the workspace and the tiling do not depend on L
    q = _plan(B, 3 * L + 17, D, N, K, **kw)
    assert q is not None
    for k in ("n_per_thread", "n_split", "seg_len", "chunk_segs", "chunk_len", "workspace_bytes"):
        assert q[k] == p[k], k


@settings(max_examples=300, deadline=None)
@given(B=st.integers(1, 4), H=st.integers(1, 64), L=st.integers(0, 1 << 20), DK=st.sampled_from([16, 32, 64]),
       DV=st.sampled_from([64, 128, 192, 256]), K=st.sampled_from([1, 2]), seg=st.sampled_from(SEGS),
       cs=st.integers(0, 64))
def test_linear_attention_plans(B, H, L, DK, DV, K, seg, cs):
    try:
        p = binding.la_plan(B, H, L, DK, DV, K, seg_len=seg, chunk_segs=cs)
    except RuntimeError as e:
        assert "INVALID_ARG" in str(e) or "UNSUPPORTED" in str(e), str(e)
        return
    assert p["workspace_bytes"] > 0 and p["chunk_len"] > 0
    assert p["chunk_len"] * max(DK, DV) <= 1 << 30
    assert p["n_chunks"] == -(-L // p["chunk_len"])
    if p["seg_len"] > 0:
        assert p["chunk_len"] == p["seg_len"] * p["chunk_segs"]
    q = binding.la_plan(B, H, 2 * L + 5, DK, DV, K, seg_len=seg, chunk_segs=cs)
    assert q["workspace_bytes"] == p["workspace_bytes"] and q["chunk_len"] == p["chunk_len"]
