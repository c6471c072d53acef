#!/usr/bin/env python3
"""Throughput of the block-quantized linear layers on one MI355X.

A step is one pass of the linear stack of one DiT denoising step: 24 blocks
at width d = 2048, each block's QKV (2048->6144), attention-out
(2048->2048), FFN-up (2048->8192) and FFN-down (8192->2048) as one grouped
qlinear_block_forward launch; q4 weights (block 32, fp16 scales,
~N(0, 0.02)), bf16 activations of 2048 tokens (2 guidance branches x 1024
latent frames, ~N(0, 1)).  Weights are quantized once on the GPU before
timing (quantization is a load-time step) and everything is resident in HBM
when the timed region starts.  The line also carries the skinny-M sweep
(int8 / q4, M in {1, 8, 32, 128}), the int8 single-block workload, the
dominant kernel's roofline position and the fp64 oracle timed on the host.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
ROT_BYTES = 512 << 20  # rotate weight copies past the 256 MB last-level cache
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_qgemm_step_q4.txt")
# the kernels one step launch runs (activation pre-pass + large-M GEMM) and
# the host code that picks and configures them; the recorded traffic is only
# valid for the sources it was measured on
KERNEL_SOURCES = ["paper_2607_08526_amd/csrc/qgemm_wide.hip", "paper_2607_08526_amd/csrc/xprep.hip",
                  "paper_2607_08526_amd/csrc/internal.h", "paper_2607_08526_amd/csrc/qlinear.hip"]


def kernel_source_hash():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-sweeps", action="store_true", help="skip the skinny/width sweeps")
    ap.add_argument("--dit-only", action="store_true",
                    help="time only the fused attention and the sequential DiT step graph "
                         "(the form the attention profile is taken with)")
    ap.add_argument("--step-only", action="store_true",
                    help="time the q4 step only (no sweeps, fp16 reference or epilogue step); "
                         "the form the counter runs profile")
    ap.add_argument("--sweeps-only", action="store_true",
                    help="run the skinny-M sweep and the int8 block only (no step, no JSON line)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target duration of the oracle's timed sample")
    ap.add_argument("--counter-points", action="store_true",
                    help="run every measured configuration a few times eagerly, each point "
                         "bracketed by marker dispatches, for rocprofv3 --pmc runs (see "
                         "--summarize-points), then exit")
    ap.add_argument("--summarize-points", nargs="+", metavar="DIR",
                    help="turn rocprofv3 --pmc runs of --counter-points (one directory per "
                         "counter set) into a per-point table and exit")
    ap.add_argument("--write-traffic", action="store_true",
                    help="with --summarize-points: also write the step launch's HBM traffic "
                         "record (the bench line's roofline.traffic)")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="per-point kernel durations of a rocprofv3 --kernel-trace run of "
                         "--counter-points, then exit")
    ap.add_argument("--summarize-stats", metavar="DIR",
                    help="print a kernel summary of a rocprofv3 --stats output dir and exit")
    return ap.parse_args()


def _csvs(d, suffix):
    import glob
    return sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))


def summarize_stats(d):
    """Kernel table of a rocprofv3 --kernel-trace --stats run."""
    import csv
    rows = []
    for p in _csvs(d, "kernel_stats.csv"):
        rows += list(csv.DictReader(open(p)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = [f"{'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10} {'total_ms':>10} {'pct':>6}  kernel"]
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "")
        short = name.split("(")[0][:90]
        out.append(f"{int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:10.2f} "
                   f"{float(r['MinNs']) / 1e3:10.2f} {float(r['MaxNs']) / 1e3:10.2f} "
                   f"{float(r['TotalDurationNs']) / 1e6:10.3f} {float(r['Percentage']):6.2f}  {short}")
    return "\n".join(out)


# ---- counter runs ------------------------------------------------------------
#
# rocprofv3 --pmc records counters per dispatch.  The counter mode runs every
# measured configuration (a "point") a few times eagerly, on distinct weight
# copies (so that no call finds its weights in the L2 or last-level cache of
# an earlier one), with a marker dispatch of `id` workgroups (libqlbench's
# mark_kernel) before and after the point's calls; the summary splits the
# dispatch list at the markers.  FETCH_SIZE and WRITE_SIZE are scaled by what
# they read for a pure 1 GiB read (read_ceiling_kernel) and a pure 1 GiB
# write (fill_kernel) of the same run.

CALIB_BYTES = 1 << 30
POINT_CALLS = 3


def counter_point_list(torch, ql, si):
    """(name, algorithmic bytes, flops, calls) per point: each call a
    closure on its own copy of the weights.  Everything is allocated before
    the first point runs."""
    import numpy as np
    dev = torch.device("cuda")
    pts = []

    def q(fmt, W, copies):
        Wd = torch.from_numpy(W).to(dev)
        c, s_ = ql.quantize(fmt, Wd)
        return [(c, s_)] + [(c.clone(), s_.clone()) for _ in range(copies - 1)]

    def xdev(X):
        return torch.from_numpy(X if X.dtype == np.float32 else X.view("int16")).to(dev)

    # cfg1, cfg2: the single-linear workloads
    for name in ("single_int8", "single_q4"):
        cfg = getattr(si, name)()
        fmt, W, X = cfg["fmt"], cfg["W"], xdev(cfg["X"])
        N, K = W.shape
        M = X.shape[0]
        Y = torch.empty((M, N), dtype=torch.float32, device=dev)
        cps = q(fmt, W, POINT_CALLS)
        wb = cps[0][0].numel() + 2 * cps[0][1].numel()
        calls = [(lambda c=c, s_=s_, X=X, Y=Y, fmt=fmt, N=N: ql.forward(fmt, X, c, s_, N, Y))
                 for c, s_ in cps]
        pts.append((f"{name} {N}x{K} M={M}", wb + X.numel() * X.element_size() + M * N * 4,
                    2.0 * M * N * K, calls))
    # cfg5: the few-row sweep
    for v, fmt, N, K in si.skinny_variants():
        cps = q(fmt, si.skinny_weight(v, N, K), POINT_CALLS)
        wb = cps[0][0].numel() + 2 * cps[0][1].numel()
        for M in si.SKINNY_M:
            X = xdev(si.skinny_activations(M, K))
            Y = torch.empty((M, N), dtype=torch.float32, device=dev)
            calls = [(lambda c=c, s_=s_, X=X, Y=Y, fmt=fmt, N=N: ql.forward(fmt, X, c, s_, N, Y))
                     for c, s_ in cps]
            pts.append((f"skinny {'int8' if fmt == ql.FMT_INT8 else 'q4'} {N}x{K} M={M}",
                        wb + M * K * 2 + M * N * 4, 2.0 * M * N * K, calls))

    # one DiT block (d = 2048) per call: grouped few-row calls, the int8
    # block and the q4 step's block at 2048 tokens, the paper's widths
    def block_point(label, fmt, Wfn, d, M, copies, seed):
        rng = np.random.default_rng(seed)
        xa = xdev(si.activations(rng, M, d, si.DT_BF16))
        xb = xdev(si.activations(rng, M, 4 * d, si.DT_BF16))
        lin = si.block_linears(d)
        Ys = [torch.empty((M, N), dtype=torch.float32, device=dev) for _, N, _ in lin]
        calls, wb = [], 0
        for cpy in range(copies):
            ents = []
            for i, (_, N, K) in enumerate(lin):
                c, s_ = ql.quantize(fmt, torch.from_numpy(Wfn(cpy, i)).to(dev))
                ents.append((fmt, xb if K == 4 * d else xa, c, s_, N, Ys[i]))
                if cpy == 0:
                    wb += c.numel() + 2 * s_.numel()
            g = ql.make_group(ents)
            calls.append(lambda g=g, ents=ents: ql.block_forward(None, group=g))
        act = M * (3 * d + 4 * d) * 2 + M * sum(N for _, N, _ in lin) * 4
        pts.append((label, wb + act, sum(2.0 * M * N * K for _, N, K in lin), calls))

    for fmt in (ql.FMT_INT8, ql.FMT_Q4):
        for M in (1, 8, 32):
            block_point(f"block d=2048 {'int8' if fmt == ql.FMT_INT8 else 'q4'} M={M} (grouped)",
                        fmt, lambda cpy, i: si.block_int8_weight(i), 2048, M, 2, 500 + M)
    block_point("block d=2048 int8 M=2048", ql.FMT_INT8, lambda cpy, i: si.block_int8_weight(i),
                2048, 2048, 2, 6)
    block_point("step block d=2048 q4 M=2048", ql.FMT_Q4, lambda cpy, i: si.step_q4_weight(cpy, i),
                2048, 2048, 2, 6)
    for w, (name, d, nblk) in enumerate(si.PAPER_WIDTHS):
        block_point(f"paper width {name} d={d} q4 M={si.PAPER_TOKENS}", ql.FMT_Q4,
                    lambda cpy, i, w=w: si.paper_weight(w, cpy, i), d, si.PAPER_TOKENS, 2,
                    900 + w)
    # the fused attention at the DiT shape (2 x 1024 tokens, 32 heads of 64),
    # read in place from a fused QKV tensor; bytes = Q, K, V read + O written
    B, T, d = 2, 1024, si.D_MODEL
    H = d // 64
    rng = np.random.default_rng(17)
    qkv = torch.from_numpy(si.f32_to_bf16_bits(rng.standard_normal((B * T, 3 * d)).astype(
        np.float32)).view(np.int16)).to(dev)
    Oa = torch.empty((B * T, d), dtype=torch.bfloat16, device=dev)
    calls = [(lambda: ql.attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], B, T, H, O=Oa))
             for _ in range(POINT_CALLS)]
    pts.append((f"attention B={B} T={T} H={H} dh=64 bf16", 4 * B * T * d * 2,
                4.0 * B * H * T * T * 64, calls))
    return pts


def counter_points(torch, ql, si):
    import ctypes
    from paper_2607_08526_amd import build as B
    lib = ctypes.CDLL(B.BENCH_LIB)
    lib.qlbench_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    lib.qlbench_fill.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_void_p]
    lib.qlbench_mark.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    stream = lambda: ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    pts = counter_point_list(torch, ql, si)
    torch.cuda.synchronize()
    buf = torch.empty(CALIB_BYTES, dtype=torch.uint8, device="cuda")
    for _ in range(2):
        if lib.qlbench_fill(ctypes.c_void_p(buf.data_ptr()), CALIB_BYTES, 1, stream()) or \
                lib.qlbench_read(ctypes.c_void_p(buf.data_ptr()), CALIB_BYTES,
                                 ctypes.c_void_p(sink.data_ptr()), stream()):
            raise RuntimeError("calibration launch failed")
    torch.cuda.synchronize()
    del buf
    for pid, (name, abytes, flops, calls) in enumerate(pts, start=1):
        if lib.qlbench_mark(pid, ctypes.c_void_p(sink.data_ptr()), stream()):
            raise RuntimeError("marker launch failed")
        for call in calls:
            call()
        if lib.qlbench_mark(pid, ctypes.c_void_p(sink.data_ptr()), stream()):
            raise RuntimeError("marker launch failed")
        torch.cuda.synchronize()
        log(f"point {pid}: {name}, {len(calls)} calls")
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "gpurun_out",
                           "counter_points.json"), "w") as f:
        json.dump([{"id": i, "name": n, "algo_bytes": b, "flops": fl, "calls": len(c)}
                   for i, (n, b, fl, c) in enumerate(pts, start=1)], f)


def _dispatches(d):
    """Per-dispatch counter records of a rocprofv3 --pmc run, in dispatch
    order: [(dispatch id, kernel, grid size, {counter: value})]."""
    import csv, collections
    recs = collections.OrderedDict()
    for p in _csvs(d, "counter_collection.csv"):
        for r in csv.DictReader(open(p)):
            key = int(r["Dispatch_Id"])
            if key not in recs:
                recs[key] = (key, r["Kernel_Name"], int(r["Grid_Size"]), {})
            recs[key][3][r["Counter_Name"]] = recs[key][3].get(r["Counter_Name"], 0.0) + \
                float(r["Counter_Value"])
    return [recs[k] for k in sorted(recs)]


def _split_points(disp):
    """{point id: [dispatches between its two markers]} and the calibration
    dispatches (before the first marker)."""
    out, calib, cur = {}, [], None
    for rec in disp:
        _, kern, grid, _ = rec
        if "mark_kernel" in kern:
            pid = grid // 64
            cur = None if cur == pid else pid
            if cur is not None:
                out[cur] = []
            continue
        if cur is not None:
            out[cur].append(rec)
        elif not out:
            calib.append(rec)
    return out, calib


SIMDS, XCDS = 1024, 8  # 256 CUs x 4 SIMDs; GRBM_GUI_ACTIVE is summed over the 8 XCDs


def _mfma_busy(c):
    """Fraction of the dispatch's cycles the matrix cores were busy, over
    every SIMD: SQ_VALU_MFMA_BUSY_CYCLES (summed over the 1024 SIMDs; 32 per
    32x32x16 f16 MFMA, the full issue time at the dense peak) over 1024 x
    the dispatch's cycles (GRBM_GUI_ACTIVE, summed over the 8 XCDs)."""
    busy, gui = c.get("SQ_VALU_MFMA_BUSY_CYCLES"), c.get("GRBM_GUI_ACTIVE")
    if not busy or not gui:
        return float("nan")
    return busy / (SIMDS * gui / XCDS)


def summarize_trace(d):
    """Per point of a --kernel-trace run of --counter-points: each kernel's
    average duration per call, and the wall time from the first kernel's
    start to the last one's end, per call."""
    import csv, collections
    rows = []
    for p in _csvs(d, "kernel_trace.csv"):
        rows += list(csv.DictReader(open(p)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    meta_p = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gpurun_out",
                          "counter_points.json")
    meta = {m["id"]: m for m in json.load(open(meta_p))}
    cur, groups = None, collections.OrderedDict()
    for r in rows:
        grid = int(r.get("Grid_Size_X", r.get("Grid_Size", "0")))
        if "mark_kernel" in r["Kernel_Name"]:
            pid = grid // 64
            cur = None if cur == pid else pid
            if cur is not None:
                groups[cur] = []
            continue
        if cur is not None:
            groups[cur].append(r)
    out = [f"{'id':>3} {'point':<44} {'us/call':>8} {'kernels (avg us per call)'}"]
    for pid, rs in groups.items():
        calls = meta[pid]["calls"]
        per = collections.OrderedDict()
        for r in rs:
            k = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0]
            k = k.replace("void ", "").replace("qlk::", "")
            per[k] = per.get(k, 0.0) + (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        span = (int(rs[-1]["End_Timestamp"]) - int(rs[0]["Start_Timestamp"])) / 1e3 / calls
        out.append(f"{pid:3d} {meta[pid]['name'][:44]:<44} {span:8.2f} " +
                   "  ".join(f"{k} {v / calls:.2f}" for k, v in per.items()))
    return "\n".join(out)


STEP_POINT = "step block d=2048 q4 M=2048"
TRAFFIC_COMMANDS = [
    "cd /tmp && export TMPDIR=/tmp",
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/gpurun_out/pmc_fetch -o fetch -- "
    "python3 $R/bench.py --counter-points",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/gpurun_out/pmc_write -o write -- "
    "python3 $R/bench.py --counter-points",
    "python3 $R/bench.py --summarize-points $R/gpurun_out/pmc_fetch $R/gpurun_out/pmc_write "
    "--write-traffic   (R = repository root)",
]


def summarize_points(dirs, write_traffic=False):
    import collections
    meta_p = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gpurun_out",
                          "counter_points.json")
    meta = {m["id"]: m for m in json.load(open(meta_p))}
    vals = collections.defaultdict(lambda: collections.defaultdict(float))
    kern = collections.defaultdict(lambda: collections.defaultdict(
        lambda: collections.defaultdict(float)))
    cal = {}
    taken = set()  # a counter read in several runs (GRBM_GUI_ACTIVE) counts from the first
    for d in dirs:
        pts, calib = _split_points(_dispatches(d))
        here = set()
        for _, k, _, c in calib:
            for cn, v in c.items():
                if cn in ("FETCH_SIZE", "WRITE_SIZE"):
                    tag = "read" if "read_ceiling" in k else "fill" if "fill_kernel" in k else None
                    if tag:
                        cal[(tag, cn)] = max(cal.get((tag, cn), 0.0), v * 1024.0)
        for pid, recs in pts.items():
            calls = meta[pid]["calls"]
            for _, k, _, c in recs:
                short = k.replace("(anonymous namespace)::", "").split("(")[0].replace("void ", "")
                for cn, v in c.items():
                    here.add(cn)
                    if cn in taken:
                        continue
                    vals[pid][cn] += v / calls
                    kern[pid][short][cn] += v / calls
        taken |= here
    fcal = cal.get(("read", "FETCH_SIZE"), 0.0) / CALIB_BYTES
    wcal = cal.get(("fill", "WRITE_SIZE"), 0.0) / CALIB_BYTES
    lines = [f"calibration: FETCH_SIZE of a pure 1 GiB read = {fcal:.4f} x its bytes; "
             f"WRITE_SIZE of a pure 1 GiB write = {wcal:.4f} x its bytes",
             f"(read of the fill: FETCH {cal.get(('fill', 'FETCH_SIZE'), 0) / CALIB_BYTES:.4f}, "
             f"write of the read: WRITE {cal.get(('read', 'WRITE_SIZE'), 0) / CALIB_BYTES:.4f})", ""]
    hdr = (f"{'id':>3} {'point':<44} {'algo_MB':>8} {'fetch_MB':>9} {'write_MB':>9} "
           f"{'hbm/algo':>8} {'mfma_busy':>9} {'valu/mfma':>9} {'lds_conf':>8}")
    lines.append(hdr)
    rows = []
    for pid in sorted(vals):
        m, v = meta[pid], vals[pid]
        fb = v.get("FETCH_SIZE", float("nan")) * 1024 / fcal if fcal else float("nan")
        wb = v.get("WRITE_SIZE", float("nan")) * 1024 / wcal if wcal else float("nan")
        mf = v.get("SQ_INSTS_MFMA", 0.0)
        mb = _mfma_busy(v)
        vpm = (v.get("SQ_INSTS_VALU", float("nan")) - mf) / mf if mf > 0 else float("nan")
        lact = v.get("SQ_ACTIVE_INST_LDS", 0.0)
        lcf = v.get("SQ_LDS_BANK_CONFLICT", float("nan")) / lact if lact > 0 else float("nan")
        rows.append({"id": pid, "point": m["name"], "algo_bytes": m["algo_bytes"],
                     "fetch_bytes": fb, "write_bytes": wb, "mfma_busy": mb, "valu_per_mfma": vpm,
                     "lds_conflict_per_active": lcf,
                     "counters": {k: round(x, 1) for k, x in v.items()}})
        lines.append(f"{pid:3d} {m['name'][:44]:<44} {m['algo_bytes'] / 1e6:8.2f} {fb / 1e6:9.2f} "
                     f"{wb / 1e6:9.2f} {(fb + wb) / m['algo_bytes']:8.2f} {mb:9.3f} {vpm:9.2f} "
                     f"{lcf:8.3f}")
    lines.append("")
    lines.append("per kernel (per call):")
    for pid in sorted(kern):
        for k, c in kern[pid].items():
            fb = c.get("FETCH_SIZE", float("nan")) * 1024 / fcal / 1e6 if fcal else float("nan")
            wb = c.get("WRITE_SIZE", float("nan")) * 1024 / wcal / 1e6 if wcal else float("nan")
            mf = c.get("SQ_INSTS_MFMA", 0.0)
            extra = ""
            if mf > 0:
                extra = (f"  mfma_busy {_mfma_busy(c):.3f}  valu/mfma "
                         f"{(c.get('SQ_INSTS_VALU', 0.0) - mf) / mf:.2f}")
            lines.append(f"{pid:3d} {k[:60]:<60} fetch {fb:8.2f} MB  write {wb:8.2f} MB{extra}  " +
                         " ".join(f"{cn}={x:.0f}" for cn, x in sorted(c.items())
                                  if cn not in ("FETCH_SIZE", "WRITE_SIZE")))
    if write_traffic:
        step = [r for r in rows if r["point"] == STEP_POINT]
        if not step or not (step[0]["fetch_bytes"] == step[0]["fetch_bytes"]) or \
                not (step[0]["write_bytes"] == step[0]["write_bytes"]):
            raise SystemExit("the step point needs both FETCH_SIZE and WRITE_SIZE runs")
        st = step[0]
        pid = st["id"]
        rec = {
            "kernel_source_sha256": kernel_source_hash(),
            "hbm_bytes_per_launch": round(st["fetch_bytes"] + st["write_bytes"]),
            "fetch_bytes_per_launch": round(st["fetch_bytes"]),
            "write_bytes_per_launch": round(st["write_bytes"]),
            "algorithmic_bytes_per_launch": st["algo_bytes"],
            "per_kernel": {k: {"fetch_bytes": round(c.get("FETCH_SIZE", 0) * 1024 / fcal),
                               "write_bytes": round(c.get("WRITE_SIZE", 0) * 1024 / wcal)}
                           for k, c in kern[pid].items()},
            "fetch_calibration": round(fcal, 4),
            "write_calibration": round(wcal, 4),
            "commands": TRAFFIC_COMMANDS,
            "notes": "One launch = one block call of the q4 step (d = 2048, 2048 tokens): the "
                     "activation pre-pass (both activation tensors, one dispatch) and the "
                     "grouped large-M GEMM, averaged over calls on two blocks' distinct weights. "
                     "FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are divided by what they read "
                     "for a pure 1 GiB read (read_ceiling_kernel: FETCH_SIZE = 0.5 x the bytes, "
                     "the counter's request unit) and a pure 1 GiB write (fill_kernel: "
                     "WRITE_SIZE = 1.0 x) in the same run.",
        }
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
    return "\n".join(lines) + "\n\nJSON " + json.dumps(
        {"fetch_calibration": fcal, "write_calibration": wcal, "points": rows})


class Step:
    """The 24-block q4 linear stack, quantized and resident on the GPU."""

    def __init__(self, torch, ql, si, keep_host_block0=True, with_f16=True):
        self.torch, self.ql = torch, ql
        dev = torch.device("cuda")
        xa, xb = si.block_activations()
        self.xa_host, self.xb_host = xa, xb
        self.xa = torch.from_numpy(xa.view("int16")).to(dev)
        self.xb = torch.from_numpy(xb.view("int16")).to(dev)
        lin = si.block_linears()
        M = xa.shape[0]
        self.Y = [torch.empty((M, N), dtype=torch.float32, device=dev) for _, N, _ in lin]
        self.blocks, self.groups = [], []
        # the same weights as fp16 (the unquantized reference format),
        # converted on the device as input preparation
        self.groups_f16, self.keep_f16 = [], []
        self.W0 = []
        self.weight_bytes = 0
        t0 = time.time()
        import concurrent.futures as cf
        jobs = [(blk, i) for blk in range(si.N_BLOCKS) for i in range(len(lin))]
        pool = cf.ThreadPoolExecutor(max_workers=8)
        gen = pool.map(lambda bi: si.step_q4_weight(*bi), jobs)  # drawn in parallel, in order
        for blk in range(si.N_BLOCKS):
            ents, ents16 = [], []
            for i, (name, N, K) in enumerate(lin):
                W = next(gen)
                if blk == 0 and keep_host_block0:
                    self.W0.append(W)
                Wd = torch.from_numpy(W).to(dev)
                codes, scales = ql.quantize(ql.FMT_Q4, Wd)
                self.weight_bytes += codes.numel() + 2 * scales.numel()
                X = self.xb if K == 4 * si.D_MODEL else self.xa
                ents.append((ql.FMT_Q4, X, codes, scales, N, self.Y[i]))
                if with_f16:
                    w16 = Wd.to(torch.float16).view(torch.int16)
                    self.keep_f16.append(w16)
                    ents16.append((ql.FMT_F16, X, w16, None, N, self.Y[i]))
                del Wd
            self.blocks.append(ents)
            self.groups.append(ql.make_group(ents))
            if with_f16:
                self.groups_f16.append(ql.make_group(ents16))
        pool.shutdown()
        torch.cuda.synchronize()
        log(f"step weights quantized on the GPU in {time.time() - t0:.1f}s "
            f"({self.weight_bytes / 1e6:.1f} MB of codes + scales)")
        self.flops_per_block = sum(2.0 * M * N * K for _, N, K in lin)
        self.flops = self.flops_per_block * si.N_BLOCKS
        self.M = M

    def run(self, events=None):
        for b, g in enumerate(self.groups):
            if events is not None:
                events[b][0].record()
            self.ql.block_forward(None, group=g)
            if events is not None:
                events[b][1].record()


def time_f16_step(torch, ql, step, steps, warmup):
    """The same step with the weights in fp16 (QL_FMT_F16), same timing
    method as the q4 step's total."""
    def run():
        for g in step.groups_f16:
            ql.block_forward(None, group=g)
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        run()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def epilogue_step(torch, ql, step, steps, warmup):
    """The q4 step with each block's layer epilogues: QKV + bias -> bf16 (the
    attention's input), out + bias added in place to an fp32 residual
    stream, FFN-up + bias -> GELU -> bf16 (FFN-down's input), FFN-down + bias
    added in place to a second residual stream (the two residual adds run
    in one grouped launch, so they target separate tensors).  Timed fused
    (qlinear_block_forward_ep) and unfused (the plain step, then the same
    epilogue as separate torch ops on its fp32 outputs)."""
    import torch.nn.functional as F
    dev = torch.device("cuda")
    M = step.M
    Ns = [e[4] for e in step.blocks[0]]
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    ydt = [torch.bfloat16, torch.float32, torch.bfloat16, torch.float32]
    acts = [ql.ACT_NONE, ql.ACT_NONE, ql.ACT_GELU, ql.ACT_NONE]
    Ye = [torch.zeros((M, N), dtype=dt, device=dev) for N, dt in zip(Ns, ydt)]
    bias = [[torch.randn(N, device=dev, generator=g) * 0.1 for N in Ns]
            for _ in step.blocks]
    groups = []
    for blk, ents in enumerate(step.blocks):
        ep = []
        for i, (fmt, X, c, sc, N, _) in enumerate(ents):
            res = Ye[i] if ydt[i] == torch.float32 else None
            ep.append((fmt, X, c, sc, N, Ye[i], bias[blk][i], acts[i], res))
        groups.append(ql.make_group_ep(ep))

    def fused():
        for gr in groups:
            ql.block_forward_ep(None, group=gr)

    def unfused():
        for blk, gr in enumerate(step.groups):
            ql.block_forward(None, group=gr)
            Y, b = step.Y, bias[blk]
            Ye[0].copy_(Y[0] + b[0])
            Ye[1].add_(Y[1] + b[1])
            Ye[2].copy_(F.gelu(Y[2] + b[2]))
            Ye[3].add_(Y[3] + b[3])

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(n):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    n = max(3, steps // 2)
    fused_ms, unfused_ms = timed(fused, n), timed(unfused, n)
    plain_ms = timed(step.run, n)
    return {
        "note": "the q4 step with each block's epilogues (QKV+bias->bf16, out+bias+residual, "
                "FFN-up+bias->GELU->bf16, FFN-down+bias+residual) fused into the output "
                "stores, against the plain step followed by the same epilogue in torch ops",
        "fused_ms_per_step": round(fused_ms, 4),
        "unfused_ms_per_step": round(unfused_ms, 4),
        "plain_ms_per_step": round(plain_ms, 4),
        "fused_overhead_pct": round(100.0 * (fused_ms / plain_ms - 1.0), 2),
        "fusion_speedup": round(unfused_ms / fused_ms, 3),
    }


def attention_bench(torch, ql, si, step):
    """The fused attention at the DiT shape (2 sequences x 1024 tokens, 32
    heads of 64), read in place from a fused QKV tensor; graph-timed, 20
    calls per replay."""
    import numpy as np
    B, T, d = 2, step.M // 2, si.D_MODEL
    H = d // 64
    rng = np.random.default_rng(17)
    qkv = torch.from_numpy(si.f32_to_bf16_bits(rng.standard_normal((B * T, 3 * d)).astype(
        np.float32)).view(np.int16)).cuda()
    O = torch.empty((B * T, d), dtype=torch.bfloat16, device="cuda")
    R = 20  # calls per graph replay: the per-call time without the replay's launch cost

    def fn():
        for _ in range(R):
            ql.attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], B, T, H, O=O)

    med = graph_time(torch, fn)[0] / R
    flops = 4.0 * B * H * T * T * 64
    tf = flops / (med * 1e-3) / 1e12
    return {"shape": f"B={B} T={T} H={H} dh=64, bf16 out", "us": round(med * 1e3, 2),
            "TFLOPs": round(tf, 1), "mfma_frac": round(tf / BF16_MFMA_PEAK_TFLOPS, 4)}


def dit_step(torch, ql, si, step):
    """A chained DiT denoising step in one HIP graph, the blocks feeding one
    another through the residual stream: per block, QKV linear (+ bias ->
    bf16) on the bf16 copy of the residual stream h, attention (-> bf16),
    out projection (+ bias) added in place into h (fp32) with a bf16 copy of
    h written by the same kernel, FFN-up (+ bias -> GELU -> bf16) on that
    copy, FFN-down (+ bias) added in place into h with its bf16 copy (the
    next block's input), and the steering injection at one block (strength
    re-read at every replay).  The first block reads a fixed h0 (out of
    place), so every replay computes the same step.  The block's
    normalizations and modulation are not part of this library.  Same q4
    weights as the step."""
    dev = torch.device("cuda")
    M, d = step.M, si.D_MODEL
    B, T, H = 2, M // 2, d // 64
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    lin = [(e[4], e[1].shape[1]) for e in step.blocks[0]]  # (N, K)
    qkv = torch.empty((M, 3 * d), dtype=torch.bfloat16, device=dev)
    att = torch.empty((M, d), dtype=torch.bfloat16, device=dev)
    up = torch.empty((M, 4 * d), dtype=torch.bfloat16, device=dev)
    h0 = torch.randn((M, d), device=dev, generator=g)
    hb0 = h0.to(torch.bfloat16)  # input preparation, outside the graph
    h = torch.empty((M, d), dtype=torch.float32, device=dev)
    hb = torch.empty((M, d), dtype=torch.bfloat16, device=dev)
    direction = torch.randn(d, device=dev, generator=g)
    direction /= direction.norm()
    strength = torch.zeros(1, dtype=torch.float32, device=dev)
    steer_block = len(step.blocks) // 2
    calls = []
    for blk, ents in enumerate(step.blocks):
        bias = [torch.randn(N, device=dev, generator=g) * 0.1 for N, _ in lin]
        (f0, _, c0, s0, N0, _), (f1, _, c1, s1, N1, _), (f2, _, c2, s2, N2, _), \
            (f3, _, c3, s3, N3, _) = ents
        st = (direction, 30.0, strength) if blk == steer_block else None
        x_in, h_prev = (hb0, h0) if blk == 0 else (hb, h)
        calls.append((
            ql.make_group_ep([(f0, x_in, c0, s0, N0, qkv, bias[0], ql.ACT_NONE, None)]),
            ql.make_group_ep([(f1, att, c1, s1, N1, h, bias[1], ql.ACT_NONE, h_prev, None, hb)]),
            ql.make_group_ep([(f2, hb, c2, s2, N2, up, bias[2], ql.ACT_GELU, None)]),
            ql.make_group_ep([(f3, up, c3, s3, N3, h, bias[3], ql.ACT_NONE, h, st, hb)]),
            bias))
    qv = qkv.view(torch.int16)

    def run():
        for g0, g1, g2, g3, _ in calls:
            ql.block_forward_ep(None, group=g0)
            ql.attention(qv[:, :d], qv[:, d:2 * d], qv[:, 2 * d:], B, T, H, O=att)
            ql.block_forward_ep(None, group=g1)
            ql.block_forward_ep(None, group=g2)
            ql.block_forward_ep(None, group=g3)

    t0 = graph_time(torch, run, reps=10, warm=3)[0]
    strength.fill_(0.15)
    t1 = graph_time(torch, run, reps=10, warm=3)[0]
    strength.zero_()
    lin_flops = step.flops
    att_flops = 4.0 * B * H * T * T * 64 * len(step.blocks)
    return {"note": "24 chained DiT blocks (QKV+bias->bf16 on the bf16 copy of the residual "
                    "stream, attention, out-proj+bias added in place into the fp32 residual with "
                    "its bf16 copy, FFN-up+bias->GELU->bf16, FFN-down+bias into the residual "
                    "with its bf16 copy, steering at one block) captured as one HIP graph; "
                    "the block's normalizations are not part of the library",
            "ms_per_step": round(t0, 4), "ms_per_step_steering_on": round(t1, 4),
            "TFLOPs": round((lin_flops + att_flops) / (t0 * 1e-3) / 1e12, 1),
            "attention_flop_share": round(att_flops / (lin_flops + att_flops), 4)}


def time_step(torch, step, steps, warmup):
    for _ in range(warmup):
        step.run()
    torch.cuda.synchronize()
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in step.groups] for _ in range(steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for s in range(steps):
        step.run(ev[s])
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start.elapsed_time(end)
    launch_ms = [a.elapsed_time(b) for row in ev for a, b in row]
    return total_ms, launch_ms, wall


_GRAPH_STREAM = []


def graph_time(torch, fn, reps=20, warm=5):
    """Capture fn() (a sequence of launches) in a HIP graph, replay it and
    return the median replay time in ms.  fn() runs once before the capture
    on the stream it is captured on (one stream for every call), so the
    library's per-stream workspace already has its size when captured."""
    if not _GRAPH_STREAM:
        _GRAPH_STREAM.append(torch.cuda.Stream())
    s = _GRAPH_STREAM[0]
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fn()
    for _ in range(warm):
        g.replay()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    ts.sort()
    return ts[len(ts) // 2], ts[0], ts[-1]


class ReadCeiling:
    """Time per call of a plain streaming read of a given number of bytes
    (libqlbench.so, built beside the library): the practical ceiling for a
    kernel that must stream one weight matrix, launch overhead included."""

    def __init__(self, torch):
        import ctypes
        from paper_2607_08526_amd import build as B
        self.torch = torch
        self.lib = ctypes.CDLL(B.BENCH_LIB)
        self.lib.qlbench_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                          ctypes.c_void_p]
        self.lib.qlbench_read.restype = ctypes.c_int
        self.sink = torch.zeros(4, dtype=torch.int32, device="cuda")

    def us_per_call(self, nbytes):
        import ctypes
        torch = self.torch
        nbytes = (nbytes + 15) // 16 * 16
        R = max(1, -(-ROT_BYTES // nbytes))
        bufs = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(R)]
        for b in bufs:
            b.fill_(1)

        def fn():
            s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
            for b in bufs:
                if self.lib.qlbench_read(ctypes.c_void_p(b.data_ptr()), nbytes,
                                         ctypes.c_void_p(self.sink.data_ptr()), s) != 0:
                    raise RuntimeError("read-ceiling launch failed")

        med, lo, hi = graph_time(torch, fn)
        del bufs
        return med / R * 1e3


def skinny_sweep(torch, ql, si):
    out = []
    dev = torch.device("cuda")
    ceiling = ReadCeiling(torch)
    for v, fmt, N, K in si.skinny_variants():
        W = si.skinny_weight(v, N, K)
        codes, scales = ql.quantize(fmt, torch.from_numpy(W).to(dev))
        wbytes = codes.numel() + 2 * scales.numel()
        R = max(1, -(-ROT_BYTES // wbytes))
        ceil_us = ceiling.us_per_call(wbytes)
        copies = [(codes.clone(), scales.clone()) for _ in range(R)]
        for M in si.SKINNY_M:
            X = torch.from_numpy(si.skinny_activations(M, K).view("int16")).to(dev)
            Y = torch.empty((M, N), dtype=torch.float32, device=dev)

            def fn():
                for c, s in copies:
                    ql.forward(fmt, X, c, s, N, Y)

            med, lo, hi = graph_time(torch, fn)
            t = med / R * 1e-3
            algo_bytes = wbytes + M * K * 2 + M * N * 4
            flops = 2.0 * M * N * K
            out.append({
                "fmt": "int8" if fmt == ql.FMT_INT8 else "q4", "N": N, "K": K, "M": M,
                "us_per_call": round(t * 1e6, 3),
                "weight_GBps": round(wbytes / t / 1e9, 1),
                "hbm_GBps": round(algo_bytes / t / 1e9, 1),
                "hbm_frac": round(algo_bytes / t / 1e9 / HBM_PEAK_GBPS, 4),
                "TFLOPs": round(flops / t / 1e12, 3),
                "rotation_copies": R,
                "read_ceiling_us": round(ceil_us, 3),
                "frac_of_read_ceiling": round(ceil_us / (t * 1e6), 4),
            })
            log(f"skinny {out[-1]}")
        del copies
        torch.cuda.empty_cache()
    return out


def block_few_rows(torch, ql, si):
    """One d = 2048 block's four linears (the int8 block workload's weights,
    quantized as int8 and as q4) at M in {1, 8, 32}: the grouped call (one
    launch streams all four matrices) against the four layers called one by
    one, each as a HIP graph over R copies of the weights (R x footprint >=
    512 MB, past the last-level cache)."""
    import numpy as np
    dev = torch.device("cuda")
    out = []
    Ws = [si.block_int8_weight(i) for i in range(4)]
    for fmt in (ql.FMT_INT8, ql.FMT_Q4):
        q = [ql.quantize(fmt, torch.from_numpy(W).to(dev)) for W in Ws]
        wbytes = sum(c.numel() + 2 * s_.numel() for c, s_ in q)
        R = max(1, -(-ROT_BYTES // wbytes))
        copies = [q] + [[(c.clone(), s_.clone()) for c, s_ in q] for _ in range(R - 1)]
        for M in (1, 8, 32):
            rng = np.random.default_rng(500 + M)
            xa = torch.from_numpy(si.activations(rng, M, 2048, si.DT_BF16).view("int16")).to(dev)
            xb = torch.from_numpy(si.activations(rng, M, 8192, si.DT_BF16).view("int16")).to(dev)
            Ys = [torch.empty((M, W.shape[0]), dtype=torch.float32, device=dev) for W in Ws]
            groups, singles = [], []
            for qq in copies:
                ents = [(fmt, xb if W.shape[1] == 8192 else xa, c, s_, W.shape[0], Y)
                        for (c, s_), W, Y in zip(qq, Ws, Ys)]
                groups.append(ql.make_group(ents))
                singles.append([ql.make_group([e]) for e in ents])

            def grouped():
                for g in groups:
                    ql.block_forward(None, group=g)

            def one_by_one():
                for gs in singles:
                    for g in gs:
                        ql.block_forward(None, group=g)

            tg = graph_time(torch, grouped)[0] / R * 1e-3
            ts = graph_time(torch, one_by_one)[0] / R * 1e-3
            algo = wbytes + M * (2048 * 3 + 8192) * 2 + 4 * M * sum(W.shape[0] for W in Ws)
            out.append({"fmt": "int8" if fmt == ql.FMT_INT8 else "q4", "d": 2048, "M": M,
                        "us_grouped": round(tg * 1e6, 2), "us_per_layer_calls": round(ts * 1e6, 2),
                        "weight_GBps": round(wbytes / tg / 1e9, 1),
                        "hbm_frac": round(algo / tg / 1e9 / HBM_PEAK_GBPS, 4),
                        "weight_MB": round(wbytes / 1e6, 2), "copies": R})
            log(f"block_few_rows {out[-1]}")
        del copies, groups, singles
        torch.cuda.empty_cache()
    return out


def block_int8(torch, ql, si):
    """One int8 block (d = 2048, 2048 tokens): a HIP graph of R block calls
    over R copies of the weights (R x 53.5 MB >= 512 MB, past the last-level
    cache, as the step's distinct blocks are), per call."""
    dev = torch.device("cuda")
    xa, xb = si.block_activations()
    xa_d = torch.from_numpy(xa.view("int16")).to(dev)
    xb_d = torch.from_numpy(xb.view("int16")).to(dev)
    q, wbytes = [], 0
    for i, (name, N, K) in enumerate(si.block_linears()):
        codes, scales = ql.quantize(ql.FMT_INT8, torch.from_numpy(si.block_int8_weight(i)).to(dev))
        wbytes += codes.numel() + 2 * scales.numel()
        q.append((codes, scales, N, K))
    R = max(1, -(-ROT_BYTES // wbytes))
    Ys = [torch.empty((xa.shape[0], N), dtype=torch.float32, device=dev) for _, _, N, _ in q]
    grps = []
    for r in range(R):
        ents = [(ql.FMT_INT8, xb_d if K == 4 * si.D_MODEL else xa_d,
                 c if r == 0 else c.clone(), s_ if r == 0 else s_.clone(), N, Y)
                for (c, s_, N, K), Y in zip(q, Ys)]
        grps.append(ql.make_group(ents))
    med = graph_time(torch, lambda: [ql.block_forward(None, group=g) for g in grps])[0] / R
    flops = sum(2.0 * xa.shape[0] * N * K for _, N, K in si.block_linears())
    t = med * 1e-3
    return {"us_per_block": round(med * 1e3, 2), "TFLOPs": round(flops / t / 1e12, 1),
            "mfma_frac": round(flops / t / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
            "weight_GBps": round(wbytes / t / 1e9, 1), "copies": R}


# non-packed fp32 VALU lane operations per second: 256 CUs x 4 SIMDs x 16
# lanes x 2.4 GHz (the published 157.3 TFLOP/s counts packed FMAs, which this
# build does not emit)
VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9
INT8_MFMA_PEAK_TOPS = 5000.0


def block_w8a8(torch, ql, si):
    """One DiT block (d = 2048, 2048 tokens) in W8A8: the per-token
    quantization of both activation tensors and the four int8 products, on
    the same int8 weights and activations as block_int8; each part timed as
    a HIP graph of R calls over R copies of the weights, per call."""
    dev = torch.device("cuda")
    xa, xb = si.block_activations()
    xa_d = torch.from_numpy(xa.view("int16")).to(dev)
    xb_d = torch.from_numpy(xb.view("int16")).to(dev)
    qa, sa = ql.quantize_act(xa_d)
    qb, sb = ql.quantize_act(xb_d)
    lin = si.block_linears()
    ws, Ys = [], []
    for i, (name, N, K) in enumerate(lin):
        ws.append(ql.quantize(ql.FMT_INT8, torch.from_numpy(si.block_int8_weight(i)).to(dev)))
        Ys.append(torch.empty((xa.shape[0], N), dtype=torch.float32, device=dev))
    wide = [K == 4 * si.D_MODEL for _, _, K in lin]
    wbytes = sum(c.numel() + 2 * s_.numel() for c, s_ in ws)
    R = max(1, -(-ROT_BYTES // wbytes))
    wcopies = [ws] + [[(c.clone(), s_.clone()) for c, s_ in ws] for _ in range(R - 1)]

    def quant():
        ql.quantize_act(xa_d, qa, sa)
        ql.quantize_act(xb_d, qb, sb)

    def gemms(w):
        for i, (_, N, K) in enumerate(lin):
            q, s_ = (qb, sb) if wide[i] else (qa, sa)
            ql.forward_w8a8(q, s_, w[i][0], w[i][1], N, Y=Ys[i])

    def both():
        for w in wcopies:
            quant()
            gemms(w)

    t_all = graph_time(torch, both)[0] / R
    t_q = graph_time(torch, lambda: [quant() for _ in range(R)])[0] / R
    t_g = graph_time(torch, lambda: [gemms(w) for w in wcopies])[0] / R
    M = xa.shape[0]
    mnk = sum(M * N * K for _, N, K in lin)
    valu_floor_us = mnk / 16 / VALU_LANE_OPS * 1e6  # cvt + FMA per output per 32-k block
    tops = 2.0 * mnk / (t_all * 1e-3) / 1e12
    return {"note": "per-token int8 activations x int8 block-32 weights: activation "
                    "quantization (both X) + 4 int8-MFMA products, same inputs as block_int8",
            "us_per_block": round(t_all * 1e3, 2), "act_quant_us": round(t_q * 1e3, 2),
            "gemm_us": round(t_g * 1e3, 2), "TOPs": round(tops, 1),
            "gemm_TOPs": round(2.0 * mnk / (t_g * 1e-3) / 1e12, 1),
            "int8_mfma_frac": round(2.0 * mnk / (t_g * 1e-3) / 1e12 / INT8_MFMA_PEAK_TOPS, 4),
            "valu_floor_us": round(valu_floor_us, 1),
            "valu_frac": round(valu_floor_us / (t_g * 1e3), 4)}


def paper_widths(torch, ql, si):
    """The paper's two DiT widths (q4, distinct weights per block) at the
    tokens of one 10 s clip: one step = every block's grouped call, timed as
    a HIP graph over R copies of the step's weights (R x footprint >= 512 MB,
    past the last-level cache)."""
    import numpy as np
    import concurrent.futures as cf
    dev = torch.device("cuda")
    out = []
    for w, (name, d, nblk) in enumerate(si.PAPER_WIDTHS):
        xa, xb = si.paper_activations(w)
        xa_d = torch.from_numpy(xa.view("int16")).to(dev)
        xb_d = torch.from_numpy(xb.view("int16")).to(dev)
        lin = si.block_linears(d)
        M = xa.shape[0]
        Ys = [torch.empty((M, N), dtype=torch.float32, device=dev) for _, N, _ in lin]
        jobs = [(blk, i) for blk in range(nblk) for i in range(len(lin))]
        with cf.ThreadPoolExecutor(max_workers=8) as pool:
            Ws = list(pool.map(lambda bi: si.paper_weight(w, *bi), jobs))
        q, wbytes = [], 0
        for W in Ws:
            c, sc = ql.quantize(ql.FMT_Q4, torch.from_numpy(W).to(dev))
            q.append((c, sc))
            wbytes += c.numel() + 2 * sc.numel()
        del Ws
        R = max(1, -(-512 * 10**6 // wbytes))
        copies = [q] + [[(c.clone(), sc.clone()) for c, sc in q] for _ in range(R - 1)]
        groups = []
        for qq in copies:
            for blk in range(nblk):
                ents = []
                for i, (_, N, K) in enumerate(lin):
                    c, sc = qq[blk * len(lin) + i]
                    ents.append((ql.FMT_Q4, xb_d if K == 4 * d else xa_d, c, sc, N, Ys[i]))
                groups.append(ql.make_group(ents))

        def fn():
            for g in groups:
                ql.block_forward(None, group=g)

        med, lo, hi = graph_time(torch, fn, reps=10, warm=3)
        t = med / R * 1e-3
        flops = nblk * sum(2.0 * M * N * K for _, N, K in lin)
        act = nblk * (M * d * 2 * 2 + sum(M * N * 4 for _, N, _ in lin))  # X read, Y written
        out.append({"name": name, "d": d, "blocks": nblk, "tokens": M, "fmt": "q4",
                    "ms_per_step": round(t * 1e3, 4), "TFLOPs": round(flops / t / 1e12, 1),
                    "mfma_frac": round(flops / t / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                    "weight_GBps": round(wbytes / t / 1e9, 1),
                    "hbm_frac": round((wbytes + act) / t / 1e9 / HBM_PEAK_GBPS, 4),
                    "copies": R})
        del groups, copies, q
        torch.cuda.synchronize()
    return out


def single_configs(torch, ql, si):
    """The two single-linear workloads (int8 1024x1024 with fp32 X 64x1024;
    q4 FFN-up 6144x1536 with bf16 X 256x1536), each as a HIP graph over R
    copies of the weights (R x footprint >= 512 MB, past the last-level
    cache), with the roofline time max(flops / peak, bytes / 8 TB/s).  fp32
    activations are contracted as three bf16 planes, so their MFMA peak is a
    third of the bf16 one."""
    dev = torch.device("cuda")
    out = []
    for name in ("single_int8", "single_q4"):
        cfg = getattr(si, name)()
        fmt, W, Xh, xdt = cfg["fmt"], cfg["W"], cfg["X"], cfg["xdt"]
        N, K = W.shape
        M = Xh.shape[0]
        X = torch.from_numpy(Xh if xdt == si.DT_F32 else Xh.view("int16")).to(dev)
        Y = torch.empty((M, N), dtype=torch.float32, device=dev)
        c, s_ = ql.quantize(fmt, torch.from_numpy(W).to(dev))
        wbytes = c.numel() + 2 * s_.numel()
        R = max(1, -(-ROT_BYTES // wbytes))
        copies = [(c, s_)] + [(c.clone(), s_.clone()) for _ in range(R - 1)]
        groups = [ql.make_group([(fmt, X, cc, ss, N, Y)]) for cc, ss in copies]

        def fn():
            for g in groups:
                ql.block_forward(None, group=g)

        t = graph_time(torch, fn)[0] / R * 1e-3
        flops = 2.0 * M * N * K
        abytes = wbytes + X.numel() * X.element_size() + M * N * 4
        peak = BF16_MFMA_PEAK_TFLOPS / (3.0 if xdt == si.DT_F32 else 1.0)
        t_roof = max(flops / (peak * 1e12), abytes / (HBM_PEAK_GBPS * 1e9))
        out.append({"workload": name, "fmt": "int8" if fmt == ql.FMT_INT8 else "q4",
                    "M": M, "N": N, "K": K, "x": "fp32" if xdt == si.DT_F32 else "bf16",
                    "us_per_call": round(t * 1e6, 3), "TFLOPs": round(flops / t / 1e12, 2),
                    "hbm_GBps": round(abytes / t / 1e9, 1),
                    "roofline_us": round(t_roof * 1e6, 3),
                    "roofline_bound": "mfma" if flops / (peak * 1e12) >= abytes / (
                        HBM_PEAK_GBPS * 1e9) else "hbm",
                    "roofline_frac": round(t_roof / t, 4), "copies": R})
        log(f"single {out[-1]}")
        del copies, groups
    return out


def host_info():
    """The host's CPU model and the cores the process may run on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0)),
            "os_cpu_count": os.cpu_count()}


class ClockSampler:
    """Samples the GPU's current graphics (shader) clock in a thread while a
    workload runs (amd-smi's Python interface, else rocm-smi)."""

    def __init__(self, period=0.02):
        import threading
        self.period, self.samples, self.source = period, [], None
        self._stop = threading.Event()
        self._read = self._setup()
        self._thread = threading.Thread(target=self._loop, daemon=True)

    def _setup(self):
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            h = amdsmi.amdsmi_get_processor_handles()[0]
            gfx = amdsmi.AmdSmiClkType.GFX

            def read():
                return float(amdsmi.amdsmi_get_clock_info(h, gfx)["clk"])
            read()
            self.source = "amdsmi gfx clock"
            return read
        except Exception:
            pass
        import re
        import subprocess

        def read_smi():
            out = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True,
                                 timeout=5).stdout
            m = re.search(r"sclk clock level:\s*\d+:\s*\((\d+)Mhz\)", out)
            return float(m.group(1)) if m else None
        try:
            if read_smi() is not None:
                self.source = "rocm-smi sclk"
                self.period = 0.2
                return read_smi
        except Exception:
            pass
        return None

    def _loop(self):
        while not self._stop.is_set():
            try:
                v = self._read()
                if v:
                    self.samples.append(v)
            except Exception:
                pass
            self._stop.wait(self.period)

    def __enter__(self):
        if self._read:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._read:
            self._thread.join()
        return False

    def summary(self):
        if not self.samples:
            return {"sclk_mhz": None, "samples": 0, "source": self.source}
        v = sorted(self.samples)
        return {"sclk_mhz": v[len(v) // 2], "sclk_mhz_min": v[0], "sclk_mhz_max": v[-1],
                "samples": len(v), "source": self.source}


def step_clock(torch, step, seconds=0.6):
    """The shader clock while the step runs back to back for ~0.6 s (the
    step's GEMMs run power-limited below the 2.4 GHz peak clock)."""
    import time as _t
    step.run()
    torch.cuda.synchronize()
    with ClockSampler() as cs:
        t0 = _t.perf_counter()
        while _t.perf_counter() - t0 < seconds:
            for _ in range(10):
                step.run()
            torch.cuda.synchronize()
    return cs.summary()


def oracle_timings(step, si):
    """The fp64 oracle timed per workload, quantization and forward apart,
    on the host cores the process may run on: the single linears and the
    few-row sweep in full, one int8 block at 2048 tokens in full, and the
    24-block q4 step as 24 x one block (quantization of block 0's weights,
    forward rate of the cpu_baseline sample), labelled extrapolated."""
    import numpy as np
    from oracle import oracle as O
    orc = O.default()
    out = {"threads": orc.num_threads(), **host_info()}

    def timed(f):
        t = time.perf_counter()
        r = f()
        return r, time.perf_counter() - t

    rows = []
    for name in ("single_int8", "single_q4"):
        cfg = getattr(si, name)()
        (cr, sr), tq = timed(lambda: orc.quantize(cfg["fmt"], cfg["W"]))
        N, K = cfg["W"].shape
        _, tf = timed(lambda: orc.forward(cfg["fmt"], cfg["X"], cfg["xdt"], cr, sr, N))
        fl = 2.0 * cfg["X"].shape[0] * N * K
        rows.append({"workload": name, "quantize_s": round(tq, 4), "forward_s": round(tf, 4),
                     "forward_GFLOPs": round(fl / tf / 1e9, 3)})
    sk_q, sk_f, sk_fl = 0.0, 0.0, 0.0
    for v, fmt, N, K in si.skinny_variants():
        W = si.skinny_weight(v, N, K)
        (cr, sr), tq = timed(lambda: orc.quantize(fmt, W))
        sk_q += tq
        for M in si.SKINNY_M:
            X = si.skinny_activations(M, K)
            _, tf = timed(lambda: orc.forward(fmt, X, O.DT_BF16, cr, sr, N))
            sk_f += tf
            sk_fl += 2.0 * M * N * K
    rows.append({"workload": "skinny sweep (4 weights x M in 1, 8, 32, 128)",
                 "quantize_s": round(sk_q, 4), "forward_s": round(sk_f, 4),
                 "forward_GFLOPs": round(sk_fl / sk_f / 1e9, 3)})
    xa, xb = step.xa_host, step.xb_host
    bq, bf, bfl = 0.0, 0.0, 0.0
    for i, (_, N, K) in enumerate(si.block_linears()):
        W = si.block_int8_weight(i)
        (cr, sr), tq = timed(lambda: orc.quantize(O.FMT_INT8, W))
        X = xb if K == 4 * si.D_MODEL else xa
        _, tf = timed(lambda: orc.forward(O.FMT_INT8, X, O.DT_BF16, cr, sr, N))
        bq, bf, bfl = bq + tq, bf + tf, bfl + 2.0 * X.shape[0] * N * K
    rows.append({"workload": "block_int8 (one d=2048 block, 2048 tokens, in full)",
                 "quantize_s": round(bq, 3), "forward_s": round(bf, 3),
                 "forward_GFLOPs": round(bfl / bf / 1e9, 3)})
    q4q = sum(timed(lambda W=W: orc.quantize(O.FMT_Q4, W))[1] for W in step.W0)
    out["rows"] = rows
    out["q4_block0_quantize_s"] = round(q4q, 3)
    return out


def cpu_baseline(step, si, target_s):
    """The fp64 oracle on a bounded sample of the same workload: rows of
    block 0's four linears (all N), after the oracle's own quantization."""
    import numpy as np
    from oracle import oracle as O
    orc = O.default()
    t0 = time.perf_counter()
    q = [orc.quantize(O.FMT_Q4, W) for W in step.W0]
    tq = time.perf_counter() - t0
    lin = si.block_linears()

    def run(rows):
        t = time.perf_counter()
        for (name, N, K), (codes, scales) in zip(lin, q):
            X = step.xb_host if K == 4 * si.D_MODEL else step.xa_host
            orc.forward(O.FMT_Q4, X, O.DT_BF16, codes, scales, N, rows=np.arange(rows))
        return time.perf_counter() - t

    # size the sample from a short run, then once more from the sample
    # itself (a one-row run overstates the per-row time)
    t1 = run(8)
    rows = int(max(1, min(step.M, 8 * target_s / max(t1, 1e-3))))
    t = run(rows)
    if t < 0.8 * target_s and rows < step.M:
        rows = int(max(1, min(step.M, rows * target_s / max(t, 1e-3))))
        t = run(rows)
    flops = rows * sum(2.0 * N * K for _, N, K in lin)
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": orc.num_threads(),
            "kind": "oracle", **host_info(), "forward_s_per_row": t / rows,
            "sample": f"fp64 oracle forward of {rows} of 2048 token rows through block 0's four "
                      f"q4 linears (all outputs), {t:.1f}s; the oracle's own quantization of "
                      f"those 50.3M weights took {tq:.2f}s (not in the rate)"}


def traffic_entry():
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    args = parse()
    if args.summarize_stats:
        print(summarize_stats(args.summarize_stats))
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.summarize_points:
        print(summarize_points(args.summarize_points, args.write_traffic))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "single-GPU benchmark: --gpus must be 1 (the multi-GPU "
                                   "sharding is a design, not implemented)"}))
        sys.exit(2)
    import torch

    import synth_inputs as si
    from paper_2607_08526_amd import qlinear as ql
    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    ql.load()

    if args.counter_points:
        counter_points(torch, ql, si)
        return

    if args.sweeps_only:
        print(json.dumps({"single_configs": single_configs(torch, ql, si),
                          "skinny": skinny_sweep(torch, ql, si),
                          "block_few_rows": block_few_rows(torch, ql, si),
                          "block_int8": block_int8(torch, ql, si),
                          "block_w8a8": block_w8a8(torch, ql, si),
                          "paper_widths": paper_widths(torch, ql, si)}), flush=True)
        return

    step = Step(torch, ql, si, keep_host_block0=not args.no_cpu_baseline,
                with_f16=not (args.step_only or args.dit_only))
    if args.dit_only:
        print(json.dumps({"attention": attention_bench(torch, ql, si, step),
                          "dit_step": dit_step(torch, ql, si, step)}), flush=True)
        return
    total_ms, launch_ms, wall = time_step(torch, step, args.steps, args.warmup)
    ms_per_step = total_ms / args.steps
    tflops = step.flops / (ms_per_step * 1e-3) / 1e12
    avg_launch_ms = sum(launch_ms) / len(launch_ms)
    achieved = step.flops_per_block / (avg_launch_ms * 1e-3) / 1e12
    log(f"step: {ms_per_step:.3f} ms, {tflops:.1f} TFLOP/s; grouped launch avg {avg_launch_ms:.4f} ms "
        f"-> {achieved:.1f} TFLOP/s; host wall {wall:.2f}s")
    clock = step_clock(torch, step)
    log(f"shader clock while the step runs: {clock}")

    res = {
        "metric": "quantized-linear TFLOP/s, one DiT denoising step's linear stack "
                  "(q4 block-32 weights, bf16 activations)",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "step_q4: 24 DiT blocks at d=2048 (QKV 2048->6144, out 2048->2048, "
                        "FFN-up 2048->8192, FFN-down 8192->2048) = 1.208B q4 weights "
                        "(block 32 along K, fp16 scales) ~N(0,0.02); bf16 activations, "
                        "2048 tokens (2 CFG branches x 1024 latent frames) ~N(0,1); "
                        "one grouped launch per block",
            "global_batch": step.M, "seq_len": 1024, "parallelism": "none (1 GPU)",
        },
        "weight_GBps": round(step.weight_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "roofline": {
            "bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / BF16_MFMA_PEAK_TFLOPS, 4),
            "traffic": traffic_entry(),
            "kernel": "one block call: xprep_kernel (bf16 -> row-shifted fp16, per distinct X) "
                      "+ qgemm_wide_kernel<q4> (fp16 MFMA, 128x256 tiles, 4 linears grouped)",
            "flops_per_launch": step.flops_per_block,
            "avg_launch_ms": round(avg_launch_ms, 5),
        },
        "sclk": clock,
    }
    if args.step_only:
        print(json.dumps(res), flush=True)
        return
    f16_ms = time_f16_step(torch, ql, step, max(3, args.steps // 2), args.warmup)
    res["fp16_reference"] = {
        "note": "the same 24-block step with the weights in fp16 (QL_FMT_F16, the "
                "unquantized reference format) through the same kernel",
        "ms_per_step": round(f16_ms, 4),
        "TFLOPs": round(step.flops / (f16_ms * 1e-3) / 1e12, 1),
        "weight_GBps": round(sum(2 * w.numel() for w in step.keep_f16) / (f16_ms * 1e-3) / 1e9, 1),
        "q4_step_speedup": round(f16_ms / ms_per_step, 3),
    }
    res["epilogue"] = epilogue_step(torch, ql, step, args.steps, args.warmup)
    res["attention"] = attention_bench(torch, ql, si, step)
    res["dit_step"] = dit_step(torch, ql, si, step)
    if not args.no_sweeps:
        res["single_configs"] = single_configs(torch, ql, si)
        res["skinny"] = skinny_sweep(torch, ql, si)
        res["block_few_rows"] = block_few_rows(torch, ql, si)
        res["block_int8"] = block_int8(torch, ql, si)
        res["block_w8a8"] = block_w8a8(torch, ql, si)
        res["paper_widths"] = paper_widths(torch, ql, si)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(step, si, args.cpu_seconds)
        ot = oracle_timings(step, si)
        per_block_fwd = res["cpu_baseline"]["forward_s_per_row"] * step.M
        ot["step_q4_extrapolated"] = {
            "note": "24 x one q4 block: the block-0 quantization time and the forward rate of "
                    "the cpu_baseline sample scaled to 2048 token rows (extrapolated, not run)",
            "quantize_s": round(24 * ot["q4_block0_quantize_s"], 2),
            "forward_s": round(24 * per_block_fwd, 1)}
        res["oracle_timings"] = ot
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
