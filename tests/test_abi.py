"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol include/pgf.h declares, plans tilings whose workspace does not
depend on L, and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2512_23068_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "pgf.h")) as f:
        txt = f.read()
    # function declarations: a return type at the start of a line, then the name
    return sorted(set(re.findall(r"^(?:int|size_t|const char \*)\s*(pgf_[a-z0-9_]+)\s*\(", txt, re.M)))


def test_library_exports_every_declared_symbol():
    lib = binding.lib()
    names = _declared_functions()
    assert set(names) == set(binding.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert binding.status_string(code).startswith("PGF_")
    assert "unknown" in binding.status_string(7)


@pytest.mark.parametrize("shape", [(1, 16, 16, 1), (1, 1536, 16, 1), (1, 5120, 16, 1), (4, 2048, 64, 8),
                                   (2, 300, 32, 2), (3, 77, 4, 4)])
def test_workspace_independent_of_L(shape):
    B, D, N, K = shape
    sizes = {binding.workspace_bytes(B, L, D, N, K) for L in (1, 1000, 8192, 16384, 32768, 65536, 131072, 1 << 22)}
    assert len(sizes) == 1 and sizes.pop() > 0
    p0 = binding.plan(B, 8192, D, N, K)
    p1 = binding.plan(B, 131072, D, N, K)
    for k in ("n_per_thread", "n_split", "seg_len", "chunk_segs", "chunk_len", "workspace_bytes"):
        assert p0[k] == p1[k], k


def test_plans_of_the_benchmark_workloads():
    p = binding.plan(1, 131072, 1536, 16, 1)
    assert p["n_per_thread"] * p["n_split"] == 16 and p["seg_len"] > 0
    assert p["chunk_len"] == p["seg_len"] * p["chunk_segs"]
    assert p["n_chunks"] == -(-131072 // p["chunk_len"])
    p = binding.plan(4, 32768, 2048, 64, 8)
    assert p["n_per_thread"] * p["n_split"] == 64
    # workspace stays a small fraction of the 19 GB IO payload
    assert p["workspace_bytes"] < 512 << 20
    p = binding.plan(1, 131072, 5120, 16, 1, in_dtype="bf16")
    assert p["workspace_bytes"] < 256 << 20


def test_tiling_overrides():
    p = binding.plan(1, 5000, 64, 16, 1, seg_len=-1)
    assert p["seg_len"] == 0
    p = binding.plan(1, 5000, 64, 16, 1, seg_len=128, chunk_segs=3)
    assert p["seg_len"] == 128 and p["chunk_segs"] == 3 and p["chunk_len"] == 384 and p["n_chunks"] == 14
    for bad in (dict(seg_len=100), dict(seg_len=8), dict(seg_len=1 << 17), dict(chunk_segs=-2),
                dict(chunk_segs=5000)):
        with pytest.raises(RuntimeError, match="INVALID_ARG"):
            binding.plan(1, 5000, 64, 16, 1, **bad)


@pytest.mark.parametrize("B,L,D,N,K,code", [
    (0, 10, 16, 16, 1, "INVALID_ARG"), (1, -1, 16, 16, 1, "INVALID_ARG"), (1, 10, 0, 16, 1, "INVALID_ARG"),
    (1, 10, 16, 0, 1, "INVALID_ARG"), (1, 10, 16, 16, 0, "INVALID_ARG"),
    (1, 10, 16, 12, 1, "UNSUPPORTED"), (1, 10, 16, 128, 1, "UNSUPPORTED"), (1, 10, 16, 16, 3, "UNSUPPORTED"),
    (1, 10, 16, 16, 9, "UNSUPPORTED")])
def test_invalid_sizes(B, L, D, N, K, code):
    assert binding.workspace_bytes(B, L, D, N, K) == 0
    with pytest.raises(RuntimeError, match=code):
        binding.plan(B, L, D, N, K)


def _call(p, x=1 << 20, dx=2 << 20, y=3 << 20, dy=4 << 20):
    """pgf_scan_jvp with fake (never dereferenced) addresses: every case here
    fails the host-side checks, which run before any HIP call."""
    lib = binding.lib()
    v = lambda a: ctypes.c_void_p(a) if a else None
    return lib.pgf_scan_jvp(v(x), v(dx), ctypes.byref(p), v(y), v(dy), None)


def _valid_params(L=100, D=16, N=16, K=1):
    p = binding.make_params(1, L, D, N, K)
    base = 1 << 30
    for i, name in enumerate(("A", "w_delta", "b_delta", "W_B", "W_C")):
        setattr(p, name, base + i * 4096)
    p.workspace_bytes = binding.lib().pgf_workspace_bytes(ctypes.byref(p))
    p.workspace = 1 << 36
    return p


def _copy_params(p):
    q = binding.PgfParams()
    ctypes.memmove(ctypes.byref(q), ctypes.byref(p), ctypes.sizeof(p))
    return q


def test_scan_rejects_bad_arguments_before_launch():
    ok = _valid_params()
    # the fake pointers above are all disjoint: only the listed defects fail
    for field in ("A", "w_delta", "b_delta", "W_B", "W_C"):
        p = _valid_params()
        setattr(p, field, None)
        assert _call(p) == -1, field
    p = _valid_params()
    p.workspace = None
    assert _call(p) == -3
    p = _valid_params()
    p.workspace_bytes -= 1
    assert _call(p) == -3
    p = _valid_params()
    p.workspace += 4          # misaligned
    assert _call(p) == -3
    assert _call(ok, x=0) == -1
    assert _call(ok, dy=0) == -1
    # y overlapping x (100*16*4 bytes each)
    assert _call(ok, x=1 << 20, y=(1 << 20) + 64) == -1
    # dy overlapping y
    assert _call(ok, y=3 << 20, dy=(3 << 20) + 128) == -1
    # the workspace overlapping an input
    assert _call(ok, x=(1 << 36) + 256) == -1
    assert _call(ok, dx=(1 << 36) - 1024) == -1
    p = _valid_params()
    p.in_dtype = 5
    assert _call(p) == -1
    p = _valid_params(N=12)
    assert _call(p) == -2


def test_binding_refuses_host_tensors_and_missing_library(monkeypatch):
    import torch
    x = torch.zeros(1, 4, 16)
    dx = torch.zeros(1, 1, 4, 16)
    with pytest.raises(ValueError, match="device tensors"):
        binding.scan_jvp(x, dx, {"A": torch.zeros(16, 16)})
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", "/nonexistent/libpgf.so")
    with pytest.raises(RuntimeError, match="not found"):
        binding.lib()


def test_parameter_flow_plans():
    """order 3 carries two sensitivity states and ignores n_dirs; the first
    and second-order entry points refuse it."""
    p1 = binding.plan(1, 131072, 1536, 16, 1, order=3)
    p8 = binding.plan(1, 131072, 1536, 16, 8, order=3)
    assert p1 == p8 and p1["n_per_thread"] == 16
    assert len({binding.workspace_bytes(1, L, 1536, 16, 1, order=3) for L in (1, 8192, 131072)}) == 1
    p64 = binding.plan(1, 100, 16, 64, 1, order=3)       # four threads per channel
    assert p64["n_per_thread"] == 16 and p64["n_split"] == 4
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        binding.plan(1, 100, 16, 16, 1, order=4)
    p = _valid_params()
    p.order = 3
    p.workspace_bytes = binding.lib().pgf_workspace_bytes(ctypes.byref(p))
    assert _call(p) == -1


def test_variant_plans_and_bad_variant_fields():
    p = binding.plan(1, 131072, 1536, 16, 1, drive="zoh", act="silu")
    assert p == binding.plan(1, 131072, 1536, 16, 1)
    for kw in (dict(K=4), dict(N=32)):
        args = dict(B=1, L=100, D=64, N=16, K=1)
        args.update(kw)
        with pytest.raises(RuntimeError, match="UNSUPPORTED"):
            binding.plan(*args.values(), drive="zoh")
    pr = binding.make_params(1, 100, 16, 16, 1)
    pr.drive = 2
    assert binding.lib().pgf_workspace_bytes(ctypes.byref(pr)) == 0
    pr.drive, pr.activation = 0, 5
    assert binding.lib().pgf_workspace_bytes(ctypes.byref(pr)) == 0


def test_linear_attention_plans():
    p0 = binding.la_plan(1, 32, 8192, 64, 64, 1)
    p1 = binding.la_plan(1, 32, 131072, 64, 64, 1)
    for k in ("seg_len", "chunk_segs", "chunk_len", "workspace_bytes"):
        assert p0[k] == p1[k], k
    assert p1["chunk_len"] == p1["seg_len"] * p1["chunk_segs"] and p1["workspace_bytes"] <= 1 << 30
    assert binding.la_plan(1, 32, 5000, 64, 64, 1, seg_len=-1)["seg_len"] == 0
    for bad in ((1, 2, 100, 48, 64, 1), (1, 2, 100, 16, 96, 1), (1, 2, 100, 16, 64, 4)):
        with pytest.raises(RuntimeError, match="UNSUPPORTED"):
            binding.la_plan(*bad)
    with pytest.raises(RuntimeError, match="INVALID_ARG"):
        binding.la_plan(1, 2, 100, 16, 64, 1, seg_len=100)


def test_linear_attention_rejects_bad_arguments_before_launch():
    """pgf_la_scan_jvp with fake (never dereferenced) addresses: overlapping
    arrays fail the host-side checks, which run before any HIP call."""
    lib = binding.lib()
    p = binding.make_la_params(1, 2, 100, 16, 64, 1)
    p.workspace_bytes = lib.pgf_la_workspace_bytes(ctypes.byref(p))
    p.workspace = 1 << 36
    v = lambda a: ctypes.c_void_p(a) if a else None

    def call(**kw):
        a = dict(q=1 << 20, k=2 << 20, v=3 << 20, g=4 << 20, dq=5 << 20, dk=6 << 20, dv=7 << 20, dg=8 << 20,
                 o=9 << 20, do=10 << 20)
        a.update(kw)
        return lib.pgf_la_scan_jvp(*(v(a[n]) for n in ("q", "k", "v", "g", "dq", "dk", "dv", "dg")),
                                   ctypes.byref(p), v(a["o"]), v(a["do"]), None)

    assert call(q=0) == -1
    assert call(o=(2 << 20) + 64) == -1            # o overlapping k
    assert call(do=(9 << 20) + 4) == -1            # do overlapping o
    assert call(g=(1 << 36) + 512) == -1           # the workspace overlapping g
    ws = p.workspace
    p.workspace = ws + 4                           # misaligned
    assert call() == -3
    p.workspace = ws


def test_complex_transition_plans():
    p = binding.make_params(1, 1000, 64, 16, 1)
    base = binding.lib().pgf_workspace_bytes(ctypes.byref(p))
    p.A_im = 1 << 30                      # any non-NULL pointer selects the complex state
    cplx = binding.lib().pgf_workspace_bytes(ctypes.byref(p))
    assert cplx > base
    for kw in (dict(order=2, n_dirs=2), dict(order=3)):
        q = binding.make_params(1, 1000, 64, 16, 1)
        q.A_im = 1 << 30
        for k, v in kw.items():
            setattr(q, k, v)
        assert binding.lib().pgf_workspace_bytes(ctypes.byref(q)) == 0, kw
    # either drive, and the output map on the real read-out, N up to 64,
    # up to eight directions
    for N, K in ((16, 2), (32, 1), (64, 2), (16, 4), (64, 8)):
        for kw in (dict(act="silu"), dict(drive="zoh"), dict(drive="zoh", act="silu")):
            q = binding.make_params(1, 1000, 64, N, K, **kw)
            q.A_im = 1 << 30
            assert binding.lib().pgf_workspace_bytes(ctypes.byref(q)) > 0, (N, kw)


def test_group_plans():
    base = binding.make_params(1, 1000, 256, 16, 1)
    g = binding.make_params(1, 1000, 256, 16, 1)
    g.n_groups = 4
    lib = binding.lib()
    assert lib.pgf_workspace_bytes(ctypes.byref(g)) > lib.pgf_workspace_bytes(ctypes.byref(base))
    for D, G in ((256, 3), (192, 2), (192, 3)):   # D/G a multiple of 64, G*N a power of two
        q = binding.make_params(1, 1000, D, 16, 1)
        q.n_groups = G
        assert lib.pgf_workspace_bytes(ctypes.byref(q)) == 0
    q = binding.make_params(1, 1000, 256, 16, 2, order=2)
    q.n_groups = 2
    assert lib.pgf_workspace_bytes(ctypes.byref(q)) == 0


def test_low_rank_plans_and_bad_fields():
    lib = binding.lib()
    base = binding.make_params(1, 1000, 256, 16, 1)
    for R in (1, 16, 48, 128):
        q = binding.make_params(1, 1000, 256, 16, 1)
        q.dt_rank = R
        # the workspace grows by z and dz_k of one host block
        assert lib.pgf_workspace_bytes(ctypes.byref(q)) > lib.pgf_workspace_bytes(ctypes.byref(base)), R
    info = binding.plan(1, 131072, 1536, 16, 1, dt_rank=48)
    assert info["workspace_bytes"] <= 2 << 30 and info["n_per_thread"] == 16 and info["n_split"] == 1
    assert info["workspace_bytes"] == binding.plan(1, 1 << 22, 1536, 16, 1, dt_rank=48)["workspace_bytes"]
    for kw in (dict(dt_rank=-1), dict(dt_rank=129)):
        q = binding.make_params(1, 1000, 256, 16, 1)
        for k, v in kw.items():
            setattr(q, k, v)
        assert lib.pgf_workspace_bytes(ctypes.byref(q)) == 0, kw
    # first order, Euler drive, one group, real A, N <= 16, K <= 2
    for args, extra in (((1, 1000, 256, 16, 2), dict(order=2)), ((1, 1000, 256, 16, 1), dict(drive="zoh")),
                        ((1, 1000, 256, 32, 1), {}), ((1, 1000, 256, 16, 4), {})):
        q = binding.make_params(*args, **extra)
        q.dt_rank = 16
        assert lib.pgf_workspace_bytes(ctypes.byref(q)) == 0, (args, extra)
    for field, val in (("n_groups", 2), ("A_im", 1 << 30)):
        q = binding.make_params(1, 1000, 256, 16, 1)
        q.dt_rank = 16
        setattr(q, field, val)
        assert lib.pgf_workspace_bytes(ctypes.byref(q)) == 0, field
    # w_delta may be NULL with the low rank; W_dx and W_dt may not
    p = _valid_params()
    p.dt_rank = 8
    p.W_dx, p.W_dt = (1 << 30) + 8 * 4096, (1 << 30) + 9 * 4096
    p.w_delta = None
    p.workspace_bytes = lib.pgf_workspace_bytes(ctypes.byref(p))
    for field in ("W_dx", "W_dt", "b_delta"):
        q = _copy_params(p)
        setattr(q, field, None)
        assert _call(q) == -1, field


def test_parameter_flows_take_the_zoh_drive_and_the_output_map_only():
    for kw in (dict(drive="zoh"), dict(act="silu"), dict(drive="zoh", act="silu")):
        binding.plan(1, 100, 256, 16, 1, order=3, **kw)
    for kw in (dict(complex_a=True), dict(groups=4), dict(dt_rank=16)):
        with pytest.raises(RuntimeError, match="UNSUPPORTED"):
            binding.plan(1, 100, 256, 16, 1, order=3, **kw)
    # the second order takes no variant
    for kw in (dict(drive="zoh"), dict(act="silu")):
        with pytest.raises(RuntimeError, match="UNSUPPORTED"):
            binding.plan(1, 100, 256, 16, 2, order=2, **kw)


def test_step_size_flows_plan():
    """delta_flows belongs to the parameter flows: every drive and output map
    with it has kernels (the planner's dry run), the workspace grows by the
    two extra state planes, and the other orders reject the flag."""
    base = binding.workspace_bytes(1, 4096, 256, 16, 1, order=3, seg_len=64)
    for kw in (dict(), dict(drive="zoh"), dict(act="silu"), dict(drive="zoh", act="silu")):
        for seg in (0, -1, 64):
            for N in (4, 8, 16):
                p = binding.plan(2, 3000, 256, N, 1, order=3, seg_len=seg, delta_flows=True, **kw)
                assert p["n_per_thread"] == N and p["n_split"] == 1
    assert binding.workspace_bytes(1, 4096, 256, 16, 1, order=3, seg_len=64, delta_flows=True) > base
    for order in (1, 2):
        with pytest.raises(RuntimeError, match="INVALID_ARG"):
            binding.plan(1, 100, 64, 16, 2, order=order, delta_flows=True)
    for N in (32, 64):   # 16 lanes per thread, two and four threads per channel
        p = binding.plan(1, 100, 64, N, 1, order=3, delta_flows=True)
        assert p["n_per_thread"] == 16 and p["n_split"] == N // 16


def test_support_matrix_has_kernels():
    """pgf_plan succeeds only when the launch sequence has a kernel for every
    step (a host-side dry run of the dispatch, the same check the entry
    points make before enqueuing anything); every combination the header
    documents as supported passes it, the others are rejected."""
    for dt in ("f32", "bf16"):
        for seg in (0, -1, 64):
            for N in (4, 8, 16, 32, 64):
                for K in (1, 2, 4, 8):
                    p = binding.plan(2, 3000, 256, N, K, in_dtype=dt, seg_len=seg)
                    assert p["n_per_thread"] * p["n_split"] == N
                    # follow-on paths: one thread per channel, N <= 16, K <= 2
                    # (the complex state: every N and K of the first order)
                    for kw in (dict(order=2), dict(order=3), dict(drive="zoh"), dict(act="silu"),
                               dict(complex_a=True), dict(complex_a=True, act="silu"),
                               dict(complex_a=True, drive="zoh"), dict(groups=4),
                               dict(dt_rank=48), dict(order=3, drive="zoh"),
                               dict(order=3, act="silu"), dict(order=3, drive="zoh", act="silu")):
                        if kw.get("order") == 2 and K != 2:
                            continue
                        ok = (kw.get("complex_a") and "order" not in kw) or kw.get("order") in (2, 3) or \
                            (N <= 16 and K <= 2)
                        if ok:
                            binding.plan(2, 3000, 256, N, K, in_dtype=dt, seg_len=seg, **kw)
                        else:
                            with pytest.raises(RuntimeError, match="UNSUPPORTED"):
                                binding.plan(2, 3000, 256, N, K, in_dtype=dt, seg_len=seg, **kw)
