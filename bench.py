"""Benchmark of the fused primal + tangent selective scan on one MI355X.

A step is one call of the whole hot path (projections, segment aggregates,
carry, scan with outputs) over one batch of seeded synthetic input already
resident in HBM.  Prints one JSON line.

Default workload: the long-range impulse-response probe, B=1 L=131072
D=1536 N=16 K=1, f32 (the L=128k workload the metric is quoted at).

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, vendor figure
FP32_VECTOR_PEAK_TFLOPS = 157.3  # MI355X fp32 vector, vendor figure
# The same units without packed FP32 (the kernels are built without it): 256
# CUs x 4 SIMDs x 16 lanes per cycle x 2 flops per fma x 2.4 GHz.
FP32_UNPACKED_PEAK_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="pulse128k")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline leg")
    ap.add_argument("--cpu-steps", type=int, default=0, help="oracle sample length (0 = auto)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the timed steps, copy 1 GiB device-to-device once (counter calibration)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="condense two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; made with "
                         "--calib-copy) into profiles/traffic_<workload>.json and exit")
    ap.add_argument("--traffic-out", default=None, help="output path of --summarize-counters")
    ap.add_argument("--order", type=int, default=1, choices=(1, 2, 3),
                    help="2: second-order flow (two directions, pgf_scan_jvp2); "
                         "3: parameter flows with gradient accumulation (pgf_param_grads)")
    ap.add_argument("--drive", default="euler", choices=("euler", "zoh"), help="input drive (first order)")
    ap.add_argument("--act", default="identity", choices=("identity", "silu"), help="output activation (first order and parameter flows)")
    ap.add_argument("--dres", action="store_true", help="add a residual weight D_res ~ N(0,1) to the output map")
    for name in ("batch", "seqlen", "d-inner", "d-state", "n-dirs"):
        ap.add_argument(f"--{name}", type=int, default=0,
                        help=f"override the workload's {name} (0 = the workload's own; the line's workload "
                             f"name then says so)")
    ap.add_argument("--delta-params", action="store_true",
                    help="parameter flows (--order 3): also the flows of w_delta and b_delta")
    ap.add_argument("--groups", type=int, default=1,
                    help="channel groups with their own B and C (first order; D/groups a multiple of 64)")
    ap.add_argument("--complex", action="store_true",
                    help="complex diagonal transition with the S4D-Lin spectrum A = -1/2 + i*pi*n (first order)")
    ap.add_argument("--lowrank", type=int, default=0,
                    help="low-rank step size of rank R (Mamba's step-size projection; first order)")
    ap.add_argument("--seg-len", type=int, default=0, help="tiling override (0 = library default)")
    ap.add_argument("--chunk-segs", type=int, default=0, help="tiling override (0 = library default)")
    return ap.parse_args()


def scan_flops_per_lane_step(K, order=1):
    """Arithmetic of the definition per (b, t, d, n) and step, counting an fma
    as 2 and exp as 1: primal Delta*A, exp, Abar*h, B*u + s, C*h' (7 with the
    shared A*s); per direction Abar*dh + (A s)*dDelta + B*p + dB*u (7) and
    dC*h' + C*dh' (4).  The mixed second-order flow adds Abar*hvw, the two
    cross-talk products A*(Abar*h_v)*dw and A*(Abar*h_w)*dv, the curvature
    (A s)*(A*dv*dw + dvw), the drive B*q + dBv*pw + dBw*pv (19) and its
    output dCv*hw + dCw*hv + C*hvw (6).  The parameter flows (order 3, no
    tangent directions) add Abar*GA + Delta*s (3), Abar*GB + u (2), gy*C (1)
    and the three accumulations (6)."""
    if order == 3:
        return 7 + 12
    return 7 + 11 * K + (25 if order == 2 else 0)


def cplx_flops_per_lane_step(K):
    """The complex transition: |Abar|, cos and sin and their product (5),
    Abar*h and A*(Abar*h) (6 + 6), the drive (2), C*Re(h') (2); per
    direction Abar*dh (6), g*dDelta (4), B*p + dB*u (3) and dC*Re(h') +
    C*Re(dh') (4)."""
    return 21 + 17 * K


SUFFIX = {1: "", 2: "-order2", 3: "-param"}
METRIC = {1: "primal+JVP scan Gtok·ch/s at L=128k", 2: "primal+JVP+second-order scan Gtok·ch/s",
          3: "primal+parameter-gradient flows Gtok·ch/s"}


COPY_BYTES = 1 << 30
KERNEL_KIND = {"k_proj": "proj", "k_la_prep": "proj", "k_carry": "carry", "k_pcarry": "carry", "k_la_carry": "carry",
               "k_gsum": "gsum", "k_state": "state_io", "k_gout": "state_io", "k_fill0": "state_io",
               "k_la_copy": "state_io"}
SCAN_SRC = "paper_2512_23068_amd/csrc/pgf_scan_kernels.h"
PLAN_SRC = "paper_2512_23068_amd/csrc/pgf_plan.cpp"
LA_SRC = "paper_2512_23068_amd/csrc/pgf_la.hip"
# Sections of the kernel source (delimited by "// ----...---- name" lines)
# whose code a run of each order executes.
TRAFFIC_SECTIONS = {
    1: ("helpers", "variants", "k_proj", "k_scan", "k_scan_sh", "k_carry", "state in/out", "dispatch"),
    2: ("helpers", "k_proj", "k_scan2", "state in/out", "dispatch"),
    3: ("helpers", "variants", "k_proj", "parameter flows", "state in/out", "dispatch"),
}


def _sections(text):
    out, name = {}, None
    for line in text.splitlines(keepends=True):
        if line.startswith("// ------"):
            name = line.strip("/- \n")
            out[name] = ""
        elif name is not None:
            out[name] += line
    return out


def _code(text):
    """The code of a C++ source: line comments, trailing blanks and empty
    lines dropped, so that editing a comment keeps a digest."""
    out = []
    for line in text.splitlines():
        i = line.find("//")
        line = (line if i < 0 else line[:i]).rstrip()
        if line:
            out.append(line)
    return "\n".join(out)


def source_digest(order=1):
    """Digest of the code (comments aside) of the kernel sections and the
    planner the counters of an order (1, 2, 3, or "la" for linear
    attention) were taken on."""
    import hashlib
    h = hashlib.sha256()
    if order == "la":
        with open(os.path.join(ROOT, LA_SRC)) as f:
            h.update(_code(f.read()).encode())
    else:
        with open(os.path.join(ROOT, SCAN_SRC)) as f:
            sec = _sections(f.read())
        for name in TRAFFIC_SECTIONS[order]:
            h.update(name.encode())
            h.update(_code(sec[name]).encode())
    with open(os.path.join(ROOT, PLAN_SRC)) as f:
        h.update(_code(f.read()).encode())
    return h.hexdigest()


def _kernel_label(name):
    import re
    base = name.split("(")[0].replace("void ", "").strip()
    if "k_scan" in base or "k_pscan" in base or "k_la_scan" in base:
        # the OUT template argument true marks the scan with outputs
        return "scan_out" if re.search(r"[<,]\s*true\s*[,>]", base) else "seg_aggregate"
    for key, lab in KERNEL_KIND.items():
        if key in base and lab:
            return lab
    return "copy" if "copyBuffer" in base else base


def summarize_counters(workload, order, fetch_csv, write_csv, out_path=None):
    import csv
    import statistics
    per = {}
    calib = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            lab = _kernel_label(r["Kernel_Name"])
            v = float(r["Counter_Value"])
            if lab == "copy":
                if v > calib.get(counter, 0.0):
                    calib[counter] = v        # the 1 GiB copy is the largest copy dispatch
                continue
            if lab in ("proj", "seg_aggregate", "carry", "gsum", "scan_out", "state_io"):
                per.setdefault(lab, {}).setdefault(counter, []).append(v)
    la = workload.startswith(("la_", "rwkv"))
    label = workload if la else workload + SUFFIX[order]
    opt = f" --order {order}" if order != 1 else ""
    out = {"workload": label, "source_sha256": source_digest("la" if la else order),
           "calibration": {"copy_bytes": COPY_BYTES, "FETCH_SIZE_KiB": calib.get("FETCH_SIZE"),
                           "WRITE_SIZE_KiB": calib.get("WRITE_SIZE"),
                           "fetch_factor": calib.get("FETCH_SIZE", 0) * 1024 / COPY_BYTES,
                           "write_factor": calib.get("WRITE_SIZE", 0) * 1024 / COPY_BYTES},
           "kernels": {}}
    for lab, c in per.items():
        f = statistics.mean(c.get("FETCH_SIZE", [0.0]))
        w = statistics.mean(c.get("WRITE_SIZE", [0.0]))
        ff = out["calibration"]["fetch_factor"] or 1.0
        wf = out["calibration"]["write_factor"] or 1.0
        out["kernels"][lab] = {"FETCH_SIZE_KiB_per_dispatch": round(f, 1), "WRITE_SIZE_KiB_per_dispatch": round(w, 1),
                               "dispatches": len(c.get("FETCH_SIZE", [])),
                               "hbm_bytes_per_dispatch": int(f * 1024 / ff + w * 1024 / wf)}
    out["commands"] = [
        f"rocprofv3 --pmc {c} --output-format csv -d gpurun_out/pmc_{label}_{c} -o pmc -- "
        f"python3 -u bench.py --workload {workload}{opt} --steps 2 --warmup 1 --no-cpu --calib-copy"
        for c in ("FETCH_SIZE", "WRITE_SIZE")]
    path = out_path or os.path.join(ROOT, "profiles", f"traffic_{label}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(path)


def committed_traffic(workload, kind, order=1):
    """HBM bytes per dispatch of `kind` from the committed counter summary,
    or None when it is missing or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != source_digest(order):
        return None
    k = t.get("kernels", {}).get(kind)
    return None if k is None else k["hbm_bytes_per_dispatch"]


class Workload:
    """What a bench run times: one step of the hot path and its accounting."""

    def __init__(self, **kw):
        self.__dict__.update(kw)


def size_overrides(args):
    """The size fields given on the command line, as ScanConfig keywords."""
    return {k: getattr(args, k) for k in ("batch", "seqlen", "d_inner", "d_state", "n_dirs")
            if getattr(args, k, 0)}


def setup_ssm(args, np, torch, binding, inputs):
    cfg = inputs.get_config(args.workload)
    over = size_overrides(args)
    if over:
        cfg = cfg.with_(**over)
    variant = args.drive != "euler" or args.act != "identity" or args.dres or args.complex or args.groups > 1 or \
        args.lowrank > 0 or args.delta_params or bool(over)
    param_variant = args.order == 3 and not (args.complex or args.groups > 1 or args.lowrank > 0)
    if args.delta_params and args.order != 3:
        print("bench.py: --delta-params belongs to the parameter flows (--order 3)", file=sys.stderr)
        sys.exit(2)
    if variant and args.order != 1 and not param_variant:
        print("bench.py: --complex/--groups/--lowrank apply to the first order only, --drive/--act/--dres to the "
              "first order and the parameter flows", file=sys.stderr)
        sys.exit(2)
    if args.order == 2:
        # two independent N(0,1) directions on the same workload shape
        cfg = cfg.with_(n_dirs=2, dx_kind="normal")
    if args.order == 3:
        # no tangent directions: an N(0,1) adjoint signal instead
        cfg = cfg.with_(n_dirs=1, dx_kind="zero")
    B, L, D, N, K = cfg.batch, cfg.seqlen, cfg.d_inner, cfg.d_state, cfg.n_dirs
    dev = torch.device("cuda:0")
    t_gen = time.time()
    inp = inputs.make_inputs(cfg)
    print(f"bench: workload {cfg.name} B={B} L={L} D={D} N={N} K={K} {cfg.in_dtype}; inputs in "
          f"{time.time() - t_gen:.1f}s", file=sys.stderr, flush=True)
    tdt = torch.bfloat16 if cfg.in_dtype == "bf16" else torch.float32
    x = torch.from_numpy(inp["x"]).to(dev).to(tdt)
    vp = inputs.variant_params({k: inp[k] for k in ("A", "w_delta", "b_delta", "W_B", "W_C")}, cfg,
                               dres=args.dres, groups=args.groups, lowrank=args.lowrank, complex_a=args.complex)
    params = {k: (torch.from_numpy(v).to(dev) if isinstance(v, np.ndarray) else v) for k, v in vp.items()}
    s_in = x.element_size()
    y = torch.empty((B, L, D), device=dev)
    if args.order == 3:
        gy = torch.from_numpy(inputs.make_adjoint(cfg)).to(dev)
        grads = tuple(torch.zeros((D, N), device=dev) for _ in range(3)) + \
            ((torch.zeros(D, device=dev),) if args.dres else ()) + \
            ((torch.zeros(D, device=dev), torch.zeros(D, device=dev)) if args.delta_params else ())
        payload = x.numel() * s_in + gy.numel() * 4 + y.numel() * 4 + sum(g.numel() * 4 for g in grads)
    else:
        dx = torch.from_numpy(inp["dx"]).to(dev).to(tdt)
        payload = x.numel() * s_in + dx.numel() * s_in + (x.numel() + dx.numel()) * 4
        dy = torch.empty((K, B, L, D), device=dev)
        outs = (y, dy)
        if args.order == 2:
            outs = outs + (torch.empty((B, L, D), device=dev),)
            payload += x.numel() * 4
    del inp
    plan = binding.plan(B, L, D, N, K, cfg.in_dtype, args.seg_len, args.chunk_segs, args.order, args.drive, args.act,
                        complex_a=args.complex, groups=args.groups, dt_rank=args.lowrank,
                        delta_flows=args.delta_params)
    ws = torch.empty(plan["workspace_bytes"], device=dev, dtype=torch.uint8)

    if args.order == 3:
        def step():
            binding.param_grads(x, gy, params, grads=grads, workspace=ws, out=y, seg_len=args.seg_len,
                                chunk_segs=args.chunk_segs, drive=args.drive, act=args.act,
                                delta_params=args.delta_params)
    else:
        fn = binding.scan_jvp2 if args.order == 2 else binding.scan_jvp
        vkw = dict(drive=args.drive, act=args.act) if args.order == 1 else {}

        def step():
            fn(x, dx, params, workspace=ws, out=outs, seg_len=args.seg_len, chunk_segs=args.chunk_segs, **vkw)

    tokch = B * L * D
    if args.order == 3:
        alg_bytes = tokch * (s_in + 4 + 4)    # read x and gy, write y
    else:
        alg_bytes = tokch * ((1 + K) * (s_in + 4) + (4 if args.order == 2 else 0))
    name = cfg.name + SUFFIX[args.order]
    return Workload(
        step=step, tokch=tokch, alg_bytes=alg_bytes, lane_steps=tokch * N,
        flops=tokch * N * (cplx_flops_per_lane_step(K) if args.complex else scan_flops_per_lane_step(K, args.order)),
        payload=payload, plan=plan, metric=METRIC[args.order],
        kernel={1: "k_scan/k_scan_sh (scan with outputs)", 2: "k_scan2 (scan with outputs)",
                3: "k_pscan (rescan with outputs and gradient sums)"}[args.order]
        if not args.complex else "k_cscan (scan with outputs)",
        traffic=None if variant else committed_traffic(name, "scan_out", args.order),
        dtype="f32" if cfg.in_dtype == "f32" else "bf16-in/f32",
        config={"workload": name + variant_suffix(args), "batch": B, "seq_len": L, "d_inner": D, "d_state": N,
                "n_dirs": 0 if args.order == 3 else K, "in_dtype": cfg.in_dtype, "parallelism": "single GPU"},
        cpu=(lambda: cpu_baseline(cfg, args.cpu_steps)) if args.order == 1 and not variant else None,
        outputs=outs if args.order == 1 and not variant else None, cfg=cfg)


def la_flops_per_lane_step(K):
    """Arithmetic of the definition per (b, h, t, i, j): alpha*S + k*v and
    q*S' (5 counting an fma as 2); per direction alpha*dS + (alpha dg)*S +
    dk*v + k*dv (7) and dq*S' + q*dS' (4)."""
    return 5 + 11 * K


def setup_la(args, np, torch, binding, inputs):
    cfg = inputs.LA_BY_NAME[args.workload]
    if args.order != 1 or args.drive != "euler" or args.act != "identity" or args.dres or size_overrides(args):
        print("bench.py: the linear-attention workloads take no --order/--drive/--act/--dres or size overrides",
              file=sys.stderr)
        sys.exit(2)
    B, H, L, DK, DV, K = cfg.batch, cfg.heads, cfg.seqlen, cfg.d_key, cfg.d_value, cfg.n_dirs
    dev = torch.device("cuda:0")
    t_gen = time.time()
    inp = inputs.make_la_inputs(cfg)
    print(f"bench: workload {cfg.name} B={B} H={H} L={L} dk={DK} dv={DV} K={K}; inputs in "
          f"{time.time() - t_gen:.1f}s", file=sys.stderr, flush=True)
    ts = [torch.from_numpy(inp[n]).to(dev) for n in ("q", "k", "v", "g", "dq", "dk", "dv", "dg")]
    del inp
    o = torch.empty((B, H, L, DV), device=dev)
    do = torch.empty((K, B, H, L, DV), device=dev)
    payload = sum(t.numel() for t in ts) * 4 + (o.numel() + do.numel()) * 4
    plan = binding.la_plan(B, H, L, DK, DV, K, args.seg_len, args.chunk_segs)
    ws = torch.empty(plan["workspace_bytes"], device=dev, dtype=torch.uint8)

    def step():
        binding.la_scan_jvp(*ts, workspace=ws, out=(o, do), seg_len=args.seg_len, chunk_segs=args.chunk_segs)

    tokch = B * L * H * DV
    # read v, dv_k and the key-side q, k, g and tangents once, write o, do_k
    alg_bytes = tokch * 4 * (2 * (1 + K)) + B * H * L * DK * 4 * (3 + 3 * K)
    return Workload(
        step=step, tokch=tokch, alg_bytes=alg_bytes, lane_steps=tokch * DK, flops=tokch * DK * la_flops_per_lane_step(K),
        payload=payload, plan=plan, metric="decaying linear attention primal+JVP Gtok·ch/s",
        kernel="k_la_scan (scan with outputs)", traffic=committed_traffic(cfg.name, "scan_out", "la"), dtype="f32",
        config={"workload": cfg.name, "batch": B, "heads": H, "seq_len": L, "d_key": DK, "d_value": DV,
                "n_dirs": K, "parallelism": "single GPU"},
        cpu=(lambda: la_cpu_baseline(cfg, args.cpu_steps)), outputs=(o, do), cfg=cfg)


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(args.workload, args.order, *args.summarize_counters, out_path=args.traffic_out)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the scan runs on one GPU (no multi-GPU mode); --gpus must be 1", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2512_23068_amd import binding, inputs

    setup = setup_la if args.workload in inputs.LA_BY_NAME else setup_ssm
    w = setup(args, np, torch, binding, inputs)
    dev = torch.device("cuda:0")
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        w.step()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    binding.timing_read()
    # Timed region: launch timing events recorded by the library on the
    # stream its kernels run on, plus whole-step events on the same stream.
    binding.timing_enable(True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        w.step()
    ev1.record()
    torch.cuda.synchronize()
    binding.timing_enable(False)
    kern = binding.timing_read()
    ms_total = ev0.elapsed_time(ev1)
    peak = torch.cuda.max_memory_allocated()
    ms_step_instrumented = ms_total / args.steps

    # The headline pass: exactly args.steps steps without per-launch events,
    # an event between consecutive steps on the stream the library launches
    # on; ms_per_step is the median of the per-step times.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        w.step()
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    ms_step = per_step[len(per_step) // 2] if len(per_step) % 2 else \
        0.5 * (per_step[len(per_step) // 2 - 1] + per_step[len(per_step) // 2])
    ms_mean = evs[0].elapsed_time(evs[-1]) / args.steps

    value = w.tokch / (ms_step * 1e-3) / 1e9
    # Dominant kernel: the scan that writes the outputs (kind 3).  Per launch
    # it performs the whole of the algorithmic IO of its block (inputs read
    # once, outputs written once) and the whole per-lane arithmetic.
    dom_name = max(kern, key=lambda k: kern[k][0])
    so_ms, so_n = kern["scan_out"]
    so_avg_ms = so_ms / max(so_n, 1)
    launches_per_step = so_n / args.steps
    bytes_per_launch = w.alg_bytes / launches_per_step
    flops_per_launch = w.flops / launches_per_step
    hbm_gbs = bytes_per_launch / (so_avg_ms * 1e-3) / 1e9
    tflops = flops_per_launch / (so_avg_ms * 1e-3) / 1e12
    roofline = {
        "kernel": w.kernel,
        "bound": "alu",
        "achieved": round(tflops, 3),
        "peak": FP32_VECTOR_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(tflops / FP32_VECTOR_PEAK_TFLOPS, 4),
        "peak_unpacked": round(FP32_UNPACKED_PEAK_TFLOPS, 2),
        "frac_unpacked": round(tflops / FP32_UNPACKED_PEAK_TFLOPS, 4),
        "traffic": w.traffic,
        "hbm_achieved_gbs": round(hbm_gbs, 1),
        "hbm_frac": round(hbm_gbs / HBM_PEAK_GBS, 4),
        "avg_launch_ms": round(so_avg_ms, 5),
        "launches_per_step": launches_per_step,
        "dominant_kind_by_time": dom_name,
    }
    kernels = {k: {"ms_per_step": round(v[0] / args.steps, 4), "launches_per_step": v[1] / args.steps}
               for k, v in kern.items()}
    plan, payload, metric, dtype, config, alg_bytes = w.plan, w.payload, w.metric, w.dtype, w.config, w.alg_bytes
    lane_steps = w.lane_steps
    cpu_fn = None if args.no_cpu else w.cpu
    # GPU outputs of the last timed step (every step writes the same values)
    outputs = getattr(w, "outputs", None)
    wcfg = getattr(w, "cfg", None)

    if args.calib_copy:
        # A plain copy of known size: what the HBM counters read for it
        # calibrates FETCH_SIZE / WRITE_SIZE against true bytes.
        del w
        torch.cuda.empty_cache()
        src = torch.ones(1 << 28, device=dev, dtype=torch.float32)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        cpu_fn = None
    cpu, parity = None, None
    if cpu_fn is not None:
        cpu, ref = cpu_fn()
        if outputs is not None:
            parity = prefix_parity(outputs, ref, np)
            if wcfg is not None and args.workload not in inputs.LA_BY_NAME:
                parity.update(tail_parity(wcfg, outputs, np, torch))

    out = {
        "metric": metric,
        "value": round(value, 3),
        "unit": "Gtok·ch/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_stats": {"median": round(ms_step, 4), "mean": round(ms_mean, 4), "min": round(per_step[0], 4),
                              "max": round(per_step[-1], 4),
                              "instrumented_mean": round(ms_step_instrumented, 4)},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic (seeded workload recipe)",
        "config": config,
        "hbm_gbs_path": round(alg_bytes / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_path": round(alg_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        # state lanes advanced per second (a lane is one (b, d, n) of the
        # recurrence, one (b, h, key, value) entry for linear attention)
        "lane_steps_g_per_s": round(lane_steps / (ms_step * 1e-3) / 1e9, 1),
        "vram": {"peak_bytes": int(peak), "payload_bytes": int(payload), "workspace_bytes": plan["workspace_bytes"],
                 "peak_minus_payload": int(peak - payload)},
        "plan": plan,
        "kernels": kernels,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity": parity,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(out), flush=True)


def variant_suffix(args):
    parts = ([args.drive] if args.drive != "euler" else []) + ([args.act] if args.act != "identity" else []) + \
        (["dres"] if args.dres else []) + (["s4dlin"] if args.complex else []) + \
        ([f"g{args.groups}"] if args.groups > 1 else []) + ([f"lr{args.lowrank}"] if args.lowrank > 0 else []) + \
        (["dparams"] if getattr(args, "delta_params", False) else []) + \
        [f"{k}{v}" for k, v in size_overrides(args).items()]
    return "".join("-" + p for p in parts)


def cpu_baseline(cfg, cpu_steps):
    """The fp64 oracle on the host cores over a prefix of the same workload
    (all channels, the first Ls steps)."""
    import numpy as np
    from oracle import oracle
    from paper_2512_23068_amd import inputs

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))

    def run(Ls):
        sub = cfg.with_(seqlen=Ls)
        inp = inputs.make_inputs(sub)
        t0 = time.perf_counter()
        y, dy, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, chunk=4096, nthreads=threads)
        return sub, time.perf_counter() - t0, (y, dy)

    if cpu_steps:
        Ls = cpu_steps
    else:   # calibrate on a short prefix, then size the sample to ~15 s
        _, t_cal, _ = run(256)
        Ls = int(max(256, min(cfg.seqlen, 256 * 15.0 / max(t_cal, 1e-3))))
    sub, dt, ref = run(Ls)
    tokch = sub.batch * Ls * sub.d_inner
    return ({"value": round(tokch / dt / 1e9, 6), "unit": "Gtok·ch/s", "cores": threads, "cpu_model": cpu_model(),
             "kind": "oracle", "lane_steps_g_per_s": round(tokch * sub.d_state / dt / 1e9, 6),
             "sample": f"{cfg.name} first {Ls} steps, all {sub.d_inner} channels, batch {sub.batch}, "
                       f"{sub.n_dirs} direction(s); fp64; {dt:.2f}s"}, ref)


def la_cpu_baseline(cfg, cpu_steps):
    """The fp64 linear-attention oracle on the host cores over a prefix of
    the same workload (all heads, the first Ls steps)."""
    from oracle import oracle
    from paper_2512_23068_amd import inputs

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    names = ("q", "k", "v", "g", "dq", "dk", "dv", "dg")

    def run(Ls):
        sub = cfg.with_(seqlen=Ls)
        inp = inputs.make_la_inputs(sub)
        t0 = time.perf_counter()
        o, do, _, _ = oracle.la_scan_jvp(*[inp[n] for n in names], nthreads=threads)
        return sub, time.perf_counter() - t0, (o, do)

    if cpu_steps:
        Ls = cpu_steps
    else:   # calibrate on a short prefix, then size the sample to ~15 s
        _, t_cal, _ = run(64)
        Ls = int(max(64, min(cfg.seqlen, 64 * 15.0 / max(t_cal, 1e-3))))
    sub, dt, ref = run(Ls)
    return ({"value": round(sub.tok_ch / dt / 1e9, 6), "unit": "Gtok·ch/s", "cores": threads,
             "cpu_model": cpu_model(), "kind": "oracle",
             "lane_steps_g_per_s": round(sub.tok_ch * sub.d_key / dt / 1e9, 6),
             "sample": f"{cfg.name} first {Ls} steps, all {sub.heads} heads, batch {sub.batch}, "
                       f"{sub.n_dirs} direction(s); fp64; {dt:.2f}s"}, ref)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _rel_l2(np, got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.linalg.norm(ref.ravel()))
    return float(np.linalg.norm((got - ref).ravel()) / (den if den > 0 else 1.0))


def prefix_parity(outputs, ref, np):
    """The timed run's outputs over the oracle's prefix (outputs at step t
    depend only on steps <= t, bit for bit), against the oracle: relative L2
    over every channel of the prefix, per output."""
    y, dy = outputs
    yo, dyo = ref
    Ls = yo.shape[-2]
    if y.dim() == 3:       # SSM: y [B,L,D], dy [K,B,L,D]
        yg, dyg = y[:, :Ls].cpu().numpy(), dy[:, :, :Ls].cpu().numpy()
        ch = y.shape[-1]
    else:                  # linear attention: o [B,H,L,dv], do [K,B,H,L,dv]
        yg, dyg = y[:, :, :Ls].cpu().numpy(), dy[:, :, :, :Ls].cpu().numpy()
        ch = y.shape[1] * y.shape[-1]
    return {"y_rel_l2": _rel_l2(np, yg, yo), "dy_rel_l2": max(_rel_l2(np, dyg[k], dyo[k]) for k in range(len(dyo))),
            "steps": int(Ls), "channels": int(ch), "reference": "fp64 oracle (the cpu_baseline run)"}


def tail_parity(cfg, outputs, np, torch, n_ch=32, n_tail=1024):
    """The last n_tail steps of the timed run's dy against the oracle over
    the whole sequence on a seeded choice of n_ch channels (the oracle runs
    any channel on its own; its projections still contract over all)."""
    from oracle import oracle
    from paper_2512_23068_amd import inputs
    y, dy = outputs
    D = cfg.d_inner
    sel = np.sort(np.random.default_rng(7).choice(D, size=min(n_ch, D), replace=False))
    idx = torch.from_numpy(sel).to(dy.device)
    dyg = dy[:, :, -n_tail:].index_select(-1, idx).cpu().numpy()
    t0 = time.perf_counter()
    inp = inputs.make_inputs(cfg)
    _, dyo, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp, channels=sel, chunk=8192)
    return {"tail_dy_rel_l2": _rel_l2(np, dyg, dyo[:, :, -n_tail:]), "tail_steps": n_tail,
            "tail_channels": int(len(sel)), "tail_oracle_s": round(time.perf_counter() - t0, 1)}


if __name__ == "__main__":
    main()
