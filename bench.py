#!/usr/bin/env python3
"""Throughput of the pruned layer-stack forward on one MI355X.

Headline workload: a 16-layer 1B-shaped causal decoder (d = 2048, 32 heads,
SwiGLU FFN 8192, RMSNorm, RoPE), 8 sequences x 2048 rows, bf16 storage,
random-init N(0, 0.02) weights and N(0, 1) hidden rows (synthetic), pruned
after layers 4, 8 and 12 -- the largest workload of the sweep. One step =
one whole stack forward over the batch (norms, projections, attention,
contribution scores, top-k, compaction), replayed as a HIP graph with every
input already in HBM.

The keep rate is swept over 1.0, 0.5, 0.25, 0.1; `value` is the throughput
at keep rate 0.5 (input tokens per second), the other points go to `sweep`
with their speedup over keep rate 1. `other_workloads` adds the same sweep,
each with its own projection roofline, for the BERT-base-shaped encoder
(3 pruning points), the paper's own schedule (Eq. 2 after every layer,
tau = 5) on a GPT-2-small-shaped causal stack at 128, 512 and 1024 rows per
sequence, a LLaMA-3-8B-shaped slice (with its decode step), a 7B-shaped
decoder slice, a ragged batch of one 7B-shaped layer with per-sequence keep
rates, and the tiny encoder the oracle runs in full.

`roofline` is reported for the kernel class with the largest share of GPU
time, the projections: algorithmic FLOPs (2 * rows * out * in per
projection) over the summed durations of the projection kernels (the GEMM
and, where K is split, its reduce), measured with HIP events on the launch
stream, against the 2.5 PFLOP/s dense bf16 MFMA peak; `traffic` is the
counter-measured HBM bytes per projection. `roofline_by_class_at_headline`
puts every kernel class against its own bound, and `measured_ceilings`
gives what the GPU sustains on a plain copy and a vendor bf16 GEMM.
`cpu_baseline` times the float64 CPU oracle on a bounded sample of the same
workload (whole sequences; sequences are independent under the method, so
a batch figure is the per-sequence rate scaled linearly).
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tokens/sec of pruned layer-stack forward vs keep_rate (1 GPU) + roofline %"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
# exp throughput: v_exp_f32 is a half-rate VALU op on gfx950 (measured over
# the whole chip: 18.6 T exp2 per second against 37.6 T fma, lane operations),
# so a wave64 takes 8 cycles: 256 CUs x 4 SIMDs x 8 exp per clock x 2.4 GHz
PEAK_EXP_PER_S = 256 * 4 * 8 * 2.4e9
HEADLINE_RATE = 0.5
# sweep key of presets whose keep rates are drawn per sequence
PER_SEQ = "per_sequence"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dec1b")
    ap.add_argument("--keep-rates", default=None, help="comma-separated sweep")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--also", default="bert,gpt2,gpt2_n128,gpt2_n1024,llama3_8b,dec7b,ragged,tiny",
                    help="comma-separated presets whose keep-rate sweeps are reported beside "
                         "the headline workload")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches instead")
    ap.add_argument("--forward-only", action="store_true",
                    help="skip the decode, backward and mark-mode legs (counter runs of the forward)")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the backward and mark-mode legs (traces of the forward and decode)")
    ap.add_argument("--cpu-seconds", type=float, default=40.0,
                    help="wall-time budget of the headline's CPU-oracle sample (0 disables every "
                         "CPU baseline)")
    ap.add_argument("--legs", default="bert",
                    help="comma-separated other workloads that also get the backward and "
                         "mark-mode legs (the headline always does)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run one plain device copy of BYTES bytes (profiled under "
                         "rocprofv3 --pmc to scale FETCH_SIZE / WRITE_SIZE) and exit")
    ap.add_argument("--summarize-pmc", nargs=4, default=None,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="turn rocprofv3 --pmc counter CSVs of this bench and of the copy "
                         "calibration into " + "profiles/gemm_traffic.json and exit")
    ap.add_argument("--copy-bytes", type=int, default=256 << 20)
    ap.add_argument("--summarize-counters", nargs=6, default=None,
                    metavar=("FETCH_CSV", "WRITE_CSV", "SQ_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV",
                             "KERNEL_STATS_CSV"),
                    help="turn rocprofv3 counter and kernel-trace files of a one-keep-rate bench "
                         "run (--keep-rates R) into a per-kernel-class table (markdown, stdout) and "
                         "exit")
    ap.add_argument("--gemm-table", action="store_true",
                    help="only time every projection shape of the workload's sweep: the shape "
                         "policy, each GEMM kernel pinned and the vendor library's plain product "
                         "(a markdown table on stdout) and exit")
    ap.add_argument("--gemm-table-pinned", type=int, default=None, help=argparse.SUPPRESS)
    return ap.parse_args()


GEMM_SRC = os.path.join(ROOT, "paper_2509_01190_amd", "csrc", "k_gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_traffic.json")
GEMM_KERNEL_TAGS = ("gemm_bf16_", "gemm_skinny_")
REDUCE_KERNEL_TAGS = ("splitk_reduce",)


def gemm_source_hash():
    import hashlib
    with open(GEMM_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def pmc_sum(csv_path, counter, name_tags):
    """Sum over dispatches (KiB for FETCH_SIZE / WRITE_SIZE) of a counter for
    the kernels whose name contains one of name_tags, and the dispatch count."""
    import csv
    import collections
    per = collections.defaultdict(float)
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter and any(g in r["Kernel_Name"] for g in name_tags):
                per[r["Dispatch_Id"]] += float(r["Counter_Value"])
    return sum(per.values()), len(per)


def summarize_pmc(args):
    """FETCH_SIZE / WRITE_SIZE of the projections of a bench run (the GEMM
    kernel -- one of the tiled kernels or the few-row kernel -- and, where K
    is split, its reduce kernel), per projection (one GEMM dispatch each), scaled by the ratio of true to counted bytes of a
    plain copy kernel."""
    f_csv, w_csv, cf_csv, cw_csv = args.summarize_pmc
    fetch_g, n_f = pmc_sum(f_csv, "FETCH_SIZE", GEMM_KERNEL_TAGS)
    write_g, n_w = pmc_sum(w_csv, "WRITE_SIZE", GEMM_KERNEL_TAGS)
    fetch_r, n_fr = pmc_sum(f_csv, "FETCH_SIZE", REDUCE_KERNEL_TAGS)
    write_r, n_wr = pmc_sum(w_csv, "WRITE_SIZE", REDUCE_KERNEL_TAGS)
    if not n_f or not n_w:
        raise SystemExit("no GEMM dispatches in the counter files")
    copy_f, n_cf = pmc_sum(cf_csv, "FETCH_SIZE", ("copyBuffer",))
    copy_w, n_cw = pmc_sum(cw_csv, "WRITE_SIZE", ("copyBuffer",))
    copy_f, copy_w = copy_f / max(n_cf, 1), copy_w / max(n_cw, 1)
    f_scale = args.copy_bytes / (copy_f * 1024.0)
    w_scale = args.copy_bytes / (copy_w * 1024.0)
    fetch_kib = (fetch_g + fetch_r) / n_f
    write_kib = (write_g + write_r) / n_w
    out = {
        "kernel": "projections: gemm_bf16_* or gemm_skinny_kernel, plus splitk_reduce_kernel where K is split "
                  "(one bench run, headline workload)",
        "workload": args.workload,
        "gemm_source_sha256_16": gemm_source_hash(),
        "gemm_dispatches": [n_f, n_w], "reduce_dispatches": [n_fr, n_wr],
        "fetch_kib_per_projection": fetch_kib, "write_kib_per_projection": write_kib,
        "reduce_share_of_bytes": (fetch_r * f_scale + write_r * w_scale)
                                 / ((fetch_g + fetch_r) * f_scale + (write_g + write_r) * w_scale),
        "copy_bytes": args.copy_bytes, "copy_fetch_kib": copy_f, "copy_write_kib": copy_w,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "hbm_bytes_per_projection": fetch_kib * 1024.0 * f_scale + write_kib * 1024.0 * w_scale,
    }
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


# kernel classes by kernel-name fragment (the timing hook's classes)
KERNEL_CLASS_TAGS = (
    ("gemm", ("gemm_bf16_", "gemm_skinny_", "gemm_valu", "splitk_reduce")),
    ("attention", ("attn_mfma", "attn_valu")),
    ("score", ("score_mfma", "score_valu")),
    ("select", ("select_kernel",)),
    ("gather", ("gather_rows", "gather_pos")),
    ("norm", ("norm_kernel",)),
)


def kernel_short(name):
    """The kernel's name with its template arguments, without namespaces,
    return type and parameter list."""
    name = name.replace("(anonymous namespace)::", "").replace("zsa::", "")
    if name.startswith("void "):
        name = name[5:]
    depth, out = 0, []
    for ch in name:
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).strip()


def kernel_class(name):
    for cls, tags in KERNEL_CLASS_TAGS:
        if any(t in name for t in tags):
            return cls
    return "misc"


def counters_by_kernel(csv_path):
    """{short kernel name: {counter: [value per dispatch]}} of a --pmc CSV."""
    import csv
    import collections
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    names, span = {}, {}
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            key = r["Dispatch_Id"]
            per[key][r["Counter_Name"]] += float(r["Counter_Value"])
            names[key] = kernel_short(r["Kernel_Name"])
            if r.get("Start_Timestamp") and r.get("End_Timestamp"):
                span[key] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    out = collections.defaultdict(lambda: collections.defaultdict(list))
    for key, cs in per.items():
        for c, v in cs.items():
            out[names[key]][c].append(v)
        if key in span:
            out[names[key]]["_duration"].append(span[key])
    return out


def summarize_counters(args):
    """Per kernel of a one-keep-rate bench run of the workload: average
    duration (kernel trace), HBM bytes per dispatch (FETCH_SIZE and
    WRITE_SIZE, scaled by what they read for a plain copy of known size),
    MFMA work and busy cycles, against the algorithmic work of its class."""
    import csv
    from paper_2509_01190_amd import workloads as W
    from paper_2509_01190_amd import zsa
    f_csv, w_csv, sq_csv, cf_csv, cw_csv, st_csv = args.summarize_counters
    p = W.PRESETS[args.workload]
    rates = ([float(r) for r in args.keep_rates.split(",")] if args.keep_rates
             else list(p.keep_rates))
    fetch = counters_by_kernel(f_csv)
    write = counters_by_kernel(w_csv)
    sq = counters_by_kernel(sq_csv)
    copy_f, n_cf = pmc_sum(cf_csv, "FETCH_SIZE", ("copyBuffer",))
    copy_w, n_cw = pmc_sum(cw_csv, "WRITE_SIZE", ("copyBuffer",))
    f_scale = args.copy_bytes / (copy_f / max(n_cf, 1) * 1024.0)
    w_scale = args.copy_bytes / (copy_w / max(n_cw, 1) * 1024.0)
    dur = {}
    with open(st_csv) as f:
        for r in csv.DictReader(f):
            dur[kernel_short(r["Name"])] = (int(r["Calls"]), float(r["AverageNs"]) * 1e-9)
    # algorithmic work of one forward at each keep rate (every rate runs the
    # same number of forwards), per class
    lens = W.lengths(p, args.seed)
    work = {}
    for rate in rates:
        counts = zsa.keep_schedule(lens, [rate] * len(lens), p.tau, len(p.prune_after))
        plan = {"counts": counts, "rows_in": [int(sum(lens))] + [int(c.sum()) for c in counts]}
        rows_in, rows_after = layer_rows(p, plan)
        w1 = class_work(p, lens, plan, rows_in, rows_after)
        w1["gemm"] = ("TFLOP/s", float(gemm_flops(p, rows_in, rows_after)))
        for k, (unit, amount) in w1.items():
            work[k] = (unit, work.get(k, (unit, 0.0))[1] + amount)
    n_pts, L = len(p.prune_after), p.n_layers
    per_fwd = {"gemm": 4 * L * len(rates), "attention": L * len(rates),
               "score": n_pts * len(rates), "select": n_pts * len(rates),
               "gather": n_pts * len(rates), "norm": 2 * L * len(rates)}
    lines = [f"workload {p.name}, keep rates {rates} (equal numbers of forwards each).",
             "",
             f"* HBM bytes = FETCH_SIZE x {f_scale:.3f} + WRITE_SIZE x {w_scale:.3f} (KiB per "
             f"dispatch, scaled by what the counters read for a plain {args.copy_bytes >> 20} MiB "
             f"copy).",
             "* MFMA FLOPs = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 (equal to 2 M N K on every "
             "GEMM dispatch).",
             "* GRBM_GUI_ACTIVE reads about 8 times the kernel's duration at the GPU clock: it "
             "sums the 8 XCDs. The clock column is GRBM_GUI_ACTIVE / 8 / duration (same run); "
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 x 1024 SIMDs), the "
             "share of SIMD cycles the matrix cores were busy at that clock.",
             "",
             "| kernel | class | calls | avg us | HBM MB / dispatch | HBM GB/s (of 8000) | "
             "MFMA TFLOP / dispatch | MFMA TFLOP/s (of 2500) | clock GHz | MFMA busy | "
             "LDS bank conflicts / LDS instr |",
             "|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    cls_tot = {}
    for name in sorted(dur, key=lambda n: -dur[n][0] * dur[n][1]):
        calls, t = dur[name]
        cls = kernel_class(name)
        fb = np.mean(fetch[name]["FETCH_SIZE"]) * 1024 * f_scale if name in fetch else float("nan")
        wb = np.mean(write[name]["WRITE_SIZE"]) * 1024 * w_scale if name in write else float("nan")
        hbm = fb + wb
        q = sq.get(name, {})
        mops = np.mean(q["SQ_INSTS_VALU_MFMA_MOPS_BF16"]) * 512 if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in q else 0.0
        grbm = np.mean(q["GRBM_GUI_ACTIVE"]) / 8 if "GRBM_GUI_ACTIVE" in q else float("nan")
        clock = grbm / np.mean(q["_duration"]) / 1e9 if "_duration" in q else float("nan")
        busy = (np.mean(q["SQ_VALU_MFMA_BUSY_CYCLES"]) / (grbm * 1024)
                if "SQ_VALU_MFMA_BUSY_CYCLES" in q and grbm > 0 else float("nan"))
        confl = (np.mean(q["SQ_LDS_BANK_CONFLICT"]) / max(np.mean(q["SQ_INSTS_LDS"]), 1.0)
                 if "SQ_LDS_BANK_CONFLICT" in q and "SQ_INSTS_LDS" in q else float("nan"))
        lines.append(f"| `{name}` | {cls} | {calls} | {t * 1e6:.2f} | {hbm / 1e6:.2f} | "
                     f"{hbm / t / 1e9:.0f} | {mops / 1e12:.4f} | {mops / t / 1e12:.0f} | "
                     f"{clock:.2f} | {busy * 100:.1f} % | {confl:.3f} |")
        c = cls_tot.setdefault(cls, [0.0, 0.0, 0.0, 0])
        c[0] += calls * t
        c[1] += calls * hbm
        c[2] += calls * mops
        c[3] += calls
    # forwards per keep rate: attention runs once per layer and forward
    att_calls = cls_tot.get("attention", [0.0, 0.0, 0.0, 0])[3]
    fwd_per_rate = att_calls / (p.n_layers * len(rates)) if att_calls else float("nan")
    lines += ["", f"Per class: the algorithmic work of the sweep's forwards ({fwd_per_rate:.0f} per "
              f"keep rate, counted from the attention dispatches) over the class's summed kernel "
              f"time:", "",
              "| class | dispatches | total ms | measured HBM MB / dispatch | algorithmic per "
              "forward sweep | achieved | of peak |",
              "|---|---:|---:|---:|---:|---:|---:|"]
    for cls, (tt, hb, mf, n) in sorted(cls_tot.items(), key=lambda kv: -kv[1][0]):
        if cls not in per_fwd or n == 0:
            continue
        unit, amount = work[cls]
        total = amount * fwd_per_rate
        if unit == "TFLOP/s":
            alg, ach, peak = f"{amount / 1e12:.3f} TFLOP", total / tt / 1e12, PEAK_BF16_TFLOPS
            ach_s = f"{ach:.0f} TFLOP/s"
        else:
            alg, ach, peak = f"{amount / 1e6:.1f} MB", total / tt / 1e9, PEAK_HBM_GBS
            ach_s = f"{ach:.0f} GB/s"
        lines.append(f"| {cls} | {n} | {tt * 1e3:.2f} | {hb / n / 1e6:.3f} | {alg} | {ach_s} | "
                     f"{ach / peak:.3f} |")
    print("\n".join(lines))


def measured_traffic(workload):
    """HBM bytes per projection from the committed counter summary, or None
    when it covers another workload or the GEMM source changed since the
    counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != gemm_source_hash() or t.get("workload") != workload:
        return None
    return t.get("hbm_bytes_per_projection")


# kernels the GEMM table pins (ZSA_GEMM_TILE values), with the shapes each takes
GEMM_PINNED = {
    2545: "w4p 256x256",
    1925: "w4p 256x192",
    1289: "persistent 128x128",
    1281: "direct-to-LDS 128x128",
}


def pinned_takes(tile, m, n, k, epi):
    """Whether a pinned kernel takes the shape (else the policy would run)."""
    if epi == 4:                                  # rotary epilogue: direct-to-LDS only
        return tile == 1281
    persist = n % 128 == 0 and k % 64 == 0 and (m + 256) * n * 2 < (1 << 31)
    if tile == 1289:
        return persist
    if tile in (2545, 1925):
        bn = 256 if tile == 2545 else 192
        return (persist and n % bn == 0 and k >= 128 and (m + 256) * k * 2 < (1 << 31)
                and n * k * 2 < (1 << 31))
    return True


def projection_shapes(p, zsa):
    """(M, N, K, epilogue) of every projection of the workload's sweep."""
    d, F = p.d_model, p.d_ff
    dec = p.kind == 1
    shapes = set()
    lens = [p.seq_len] * p.batch
    for rate in p.keep_rates:
        counts = zsa.keep_schedule(lens, [rate] * p.batch, p.tau, len(p.prune_after))
        rows = [sum(lens)] + [int(c.sum()) for c in counts]
        point = 0
        for l in range(1, p.n_layers + 1):
            t_in = rows[point]
            if point < len(p.prune_after) and p.prune_after[point] == l:
                point += 1
            t_out = rows[point]
            shapes.add((t_in, qkv_n(p), d, 4 if dec else 0))
            shapes.add((t_out, d, d, 3))
            shapes.add((t_out, 2 * F if dec else F, d, 2 if dec else 1))
            shapes.add((t_out, d, F, 3))
    return sorted(shapes, key=lambda t: (-t[0], t[2], t[1]))


def time_projection(torch, zsa, dev, m, n, k, epi, p, split, blas=False):
    """Microseconds per projection (all its launches): minimum over six
    blocks of 40 calls, HIP events on the current stream."""
    g = torch.Generator(device="cpu").manual_seed(m * 7 + n * 3 + k)
    x = (torch.randn(m, k, generator=g) * 0.5).to(torch.bfloat16).to(dev)
    w = (torch.randn(n, k, generator=g) * 0.02).to(torch.bfloat16).to(dev)
    if blas:
        wt = w.t()
        fn = lambda: torch.matmul(x, wt)
    else:
        bias = ((torch.randn(n, generator=g) * 0.02).to(torch.bfloat16).to(dev)
                if p.kind == 0 else None)
        ncols = n // 2 if epi == 2 else n
        y = torch.empty(m, ncols, dtype=torch.bfloat16, device=dev)
        res = y.normal_() if epi == 3 else None
        pos = torch.arange(m, dtype=torch.int32, device=dev) % p.seq_len if epi == 4 else None
        hd = p.d_model // p.n_heads
        # the split-K partials, and for the rotary epilogue room for its table
        need = zsa.linear_workspace_size(zsa.BF16, m, n, k) if split else 0
        if split and epi == 4:
            need = (need + 255) // 256 * 256 + m * hd * 4
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev) if need else None
        # rotary: the q and k columns of the fused projection
        fn = lambda: zsa.linear(x, w, bias, epi, res, pos, hd, p.d_model + p.kv_heads * hd
                                if epi == 4 else 0, p.rope_theta, out=y, split=split, ws=ws)
    for _ in range(5):
        fn()
    best = None
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(6):
        e0.record()
        for _ in range(40):
            fn()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / 40
        best = us if best is None else min(best, us)
    return best


def gemm_table(args, torch, W, zsa, dev):
    """The projection shapes of a workload's sweep, timed under the shape
    policy (split K allowed), each kernel pinned (each in a child process:
    the pin is read once per process), and hipBLASLt's plain product (no
    bias, activation or residual)."""
    import subprocess
    p = W.PRESETS[args.workload]
    shapes = projection_shapes(p, zsa)
    if args.gemm_table_pinned is not None:
        tile = args.gemm_table_pinned
        out = {f"{m}x{n}x{k}x{e}": (time_projection(torch, zsa, dev, m, n, k, e, p, split=False)
                                   if pinned_takes(tile, m, n, k, e) else None)
               for m, n, k, e in shapes}
        print(json.dumps(out))
        return
    policy = {(m, n, k, e): time_projection(torch, zsa, dev, m, n, k, e, p, split=True)
              for m, n, k, e in shapes}
    blas = {(m, n, k, e): time_projection(torch, zsa, dev, m, n, k, e, p, split=False, blas=True)
            for m, n, k, e in shapes}
    pinned = {}
    for tile in GEMM_PINNED:
        env = dict(os.environ, ZSA_GEMM_TILE=str(tile))
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--workload", p.name,
                            "--gemm-table", "--gemm-table-pinned", str(tile)],
                           env=env, capture_output=True, text=True, timeout=600)
        if r.returncode != 0:
            raise SystemExit(f"pinned run {tile} failed: {r.stderr[-2000:]}")
        pinned[tile] = json.loads(r.stdout.strip().splitlines()[-1])
    epi_name = {0: "bias", 1: "GELU", 2: "SwiGLU", 3: "residual", 4: "rotary"}
    lines = [f"us per projection (all its launches; minimum of six 40-call blocks), "
             f"workload {p.name}, every projection shape of its keep-rate sweep "
             f"{list(p.keep_rates)}; `bench.py --workload {p.name} --gemm-table`.",
             "",
             "| M x N x K (epilogue) | policy | " + " | ".join(GEMM_PINNED.values())
             + " | hipBLASLt (plain) | policy TFLOP/s |",
             "|---|---:|" + "---:|" * len(GEMM_PINNED) + "---:|---:|"]
    tot_pol = tot_blas = 0.0
    for key in shapes:
        m, n, k, e = key
        pol = policy[key]
        tot_pol += pol
        tot_blas += blas[key]
        cells = []
        for tile in GEMM_PINNED:
            v = pinned[tile][f"{m}x{n}x{k}x{e}"]
            cells.append("—" if v is None else f"{v:.1f}")
        lines.append(f"| {m} x {n} x {k} ({epi_name[e]}) | **{pol:.1f}** | " + " | ".join(cells)
                     + f" | {blas[key]:.1f} | {2 * m * n * k / (pol * 1e-6) / 1e12:.0f} |")
    lines.append(f"| sum | **{tot_pol:.1f}** |" + " |" * len(GEMM_PINNED)
                 + f" {tot_blas:.1f} | |")
    print("\n".join(lines))


def qkv_n(p):
    """Output width of the fused [q | k | v] projection."""
    return p.d_model + 2 * p.kv_heads * (p.d_model // p.n_heads)


def gemm_flops(p, rows_in, rows_after):
    """Algorithmic FLOPs of the projections of each layer: 2 * M * N * K,
    with M the rows the GEMM processes (the pruned rows after the pruning
    layer's attention)."""
    d, F = p.d_model, p.d_ff
    up_n = 2 * F if p.kind == 1 else F
    total = 0
    for l in range(p.n_layers):
        t_in, t_out = rows_in[l], rows_after[l]
        total += 2 * t_in * qkv_n(p) * d       # QKV (fused; grouped-query k/v)
        total += 2 * t_out * d * d             # output projection
        total += 2 * t_out * up_n * d          # up (or gate|up)
        total += 2 * t_out * d * F             # down
    return total


def gemm_bytes(p, results, rates):
    """Algorithmic HBM bytes of the projections over the sweep: each operand
    read once, the output written once, the residual read once."""
    d, F = p.d_model, p.d_ff
    e = 2 if p.dtype == "bf16" else 4
    up_n = 2 * F if p.kind == 1 else F
    up_out = F
    total = 0
    for r in rates:
        rows_in, rows_after = results[r]["rows"]
        for l in range(p.n_layers):
            t_in, t_out = rows_in[l], rows_after[l]
            total += e * (t_in * d + qkv_n(p) * d + t_in * qkv_n(p))            # QKV
            total += e * (t_out * d + d * d + 2 * t_out * d)                    # O + residual
            total += e * (t_out * d + up_n * d + t_out * up_out)                # up
            total += e * (t_out * F + d * F + 2 * t_out * d)                    # down + residual
    return total


def class_work(p, lens, plan, rows_in, rows_after):
    """Algorithmic work per kernel class for one forward: FLOPs for the MFMA
    classes, bytes for the memory-bound ones (the per-row or per-pair figure
    times the rows or pairs each launch processes)."""
    d, H, hd, F = p.d_model, p.n_heads, p.d_model // p.n_heads, p.d_ff
    e = 2 if p.dtype == "bf16" else 4
    attn_flops = 0.0
    score_flops = 0.0
    norm_bytes = 0.0
    # per-sequence lengths through the schedule
    counts = [list(lens)] + [list(c) for c in plan["counts"]]
    point = 0
    cur = counts[0]
    for l in range(1, p.n_layers + 1):
        # Eq. 1 attention: QK^T and PV, 2*n*hd each per query and head
        # (half of that under the causal mask)
        frac = 0.5 if p.causal else 1.0
        attn_flops += sum(4.0 * n * n * hd * H * frac for n in cur)
        norm_bytes += 2.0 * rows_in[l - 1] * d * e + 2.0 * rows_after[l - 1] * d * e
        if point < len(p.prune_after) and p.prune_after[point] == l:
            # a point that keeps every row runs no score sweep (zsa_stack_forward)
            if counts[point + 1] != counts[point]:
                score_flops += sum(2.0 * n * n * hd * H * frac for n in cur)
            point += 1
            cur = counts[point]
    gather_bytes = 0.0
    select_bytes = 0.0
    for pt in range(len(p.prune_after)):
        if counts[pt + 1] == counts[pt]:  # every row kept: no selection or gather
            continue
        t_in = plan["rows_in"][pt]
        t_out = plan["rows_in"][pt + 1]
        # two row arrays (residual, attention output) read and written, plus
        # index and position words
        gather_bytes += 2 * 2.0 * t_out * d * e + 12.0 * t_out
        # scores (one partial per head group; counted as one vector) and kept rows
        select_bytes += 4.0 * t_in + 4.0 * t_out
    return {"attention": ("TFLOP/s", attn_flops), "score": ("TFLOP/s", score_flops),
            "norm": ("GB/s", norm_bytes), "gather": ("GB/s", gather_bytes),
            "select": ("GB/s", select_bytes)}


def layer_rows(p, plan):
    rows_in, rows_after = [], []
    cur = plan["rows_in"][0]
    point = 0
    for l in range(1, p.n_layers + 1):
        rows_in.append(cur)
        if point < len(p.prune_after) and p.prune_after[point] == l:
            cur = plan["rows_in"][point + 1]
            point += 1
        rows_after.append(cur)
    return rows_in, rows_after


def cpu_info():
    """Host cores visible to this process and the CPU model."""
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        affinity = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return affinity, model


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return 1


def cpu_baseline(p, ws_np, x_np, lens, rates, seqs, max_runs, budget_s):
    """The float64 oracle (as it stands, exact mode) on a bounded sample:
    the sequences ``seqs`` of the workload, run up to ``max_runs`` times
    while the budget lasts; tokens/s of each run, the median reported.
    Sequences are independent under the method, so the rate over whole
    sequences is the batch rate scaled linearly."""
    from oracle import zsa_oracle as O
    from paper_2509_01190_amd import workloads as W
    ocfg = O.LayerCfg(p.kind, p.d_model, p.n_heads, p.d_ff, p.causal, p.norm_eps, p.rope_theta,
                      p.tau, p.n_kv_heads, p.force_keep_last)
    ows = [{k: (None if v is None else W.as_f64(W.to_storage(v, p.dtype))) for k, v in w.items()}
           for w in ws_np]
    x64 = W.as_f64(W.to_storage(x_np, p.dtype))
    cu = W.cu_seqlens(lens)
    rows = int(sum(lens[b] for b in seqs))
    runs = []
    t_start = time.perf_counter()
    while len(runs) < max_runs:
        t0 = time.perf_counter()
        for b in seqs:
            n = lens[b]
            O.stack_forward(x64[cu[b]:cu[b + 1]], np.arange(n), [0, n], ows, ocfg, p.prune_after,
                            [float(rates[b])])
        runs.append(time.perf_counter() - t0)
        spent = time.perf_counter() - t_start
        if spent + runs[-1] > budget_s:
            break
    med = float(np.median(runs))
    affinity, model = cpu_info()
    rate_txt = (f"keep rate {float(rates[seqs[0]])}" if len(set(float(rates[b]) for b in seqs)) == 1
                else "per-sequence keep rates " + ", ".join(f"{float(rates[b]):.3f}" for b in seqs))
    return {"value": rows / med, "unit": "tokens/s", "cores": int(blas_threads()),
            "kind": "oracle",
            "sample": f"{len(seqs)} of {len(lens)} sequences ({rows} rows), {rate_txt}, float64 "
                      f"exact mode, median of {len(runs)} run(s) of "
                      f"{', '.join(f'{r:.1f}' for r in runs)} s; batch rate = per-sequence rate "
                      f"scaled linearly",
            "affinity_cores": affinity, "cpu_model": model}


def graph_ms(fn, args, torch):
    """Mean time of fn replayed as a HIP graph (after warm-up replays)."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fn()
    torch.cuda.current_stream().wait_stream(s)
    for _ in range(args.warmup):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        g.replay()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / args.steps


def measure(p, rates, args, torch, W, zsa, dev, timing, legs=False):
    """Graph-replayed step time of preset ``p`` at every keep rate (the mean
    over the timed replays, and the median, p10 and p90 of the per-replay
    event times), with ``timing`` the per-class launch durations of one eager
    forward, and with ``legs`` the backward and the same stack in mark-only
    mode (rows marked instead of removed)."""
    lens = W.lengths(p, args.seed)
    ws_np = W.stack_weights(p, args.seed)
    x_np = W.hidden(p, args.seed, lens)
    # float32 -> bf16 (nearest-even) on the GPU: the same numbers as the CPU
    # conversion the oracle's copy goes through, without its host time
    store = torch.bfloat16 if p.dtype == "bf16" else torch.float32
    dws = [{k: (None if v is None else torch.from_numpy(v).to(dev).to(store)) for k, v in w.items()}
           for w in ws_np]
    cfg = zsa.make_cfg(p.kind, p.d_model, p.n_heads, p.d_ff, p.causal,
                       zsa.BF16 if p.dtype == "bf16" else zsa.F32, p.tau, p.norm_eps, p.rope_theta,
                       p.n_kv_heads, p.force_keep_last)
    stack = zsa.Stack(cfg, dws)
    mcfg = zsa.make_cfg(p.kind, p.d_model, p.n_heads, p.d_ff, p.causal,
                        zsa.BF16 if p.dtype == "bf16" else zsa.F32, p.tau, p.norm_eps,
                        p.rope_theta, p.n_kv_heads, p.force_keep_last, mark_only=True)
    mstack = zsa.Stack(mcfg, dws)
    seqs = zsa.Seqs(lens, dev)
    xd = W.to_storage(x_np, p.dtype).to(dev)
    posd = torch.from_numpy(W.positions(lens)).to(dev)
    tokens = int(sum(lens))

    results = {}
    for rate in rates:
        kr = W.keep_rates(p, args.seed, None if rate == PER_SEQ else rate)
        outs = stack.forward(xd, posd, seqs, p.prune_after, kr)   # allocates outputs once
        torch.cuda.synchronize()
        if args.no_graph:
            def step():
                stack.forward(xd, posd, seqs, p.prune_after, kr, out=outs)
        else:
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                with torch.cuda.graph(g, stream=s):
                    stack.forward(xd, posd, seqs, p.prune_after, kr, out=outs)
            torch.cuda.current_stream().wait_stream(s)
            step = g.replay
        for _ in range(args.warmup):
            step()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for a, b in evs:
            a.record()
            step()
            b.record()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        per = np.array([a.elapsed_time(b) for a, b in evs])
        plan = stack.plan(seqs, p.prune_after, kr)
        r = {"ms": ms, "tok_s": tokens / (ms * 1e-3), "kept_rows_final": plan["final_rows"],
             "step_ms": {"median": float(np.median(per)), "p10": float(np.percentile(per, 10)),
                         "p90": float(np.percentile(per, 90))}}
        if p.causal and p.force_keep_last and not args.forward_only:
            r["decode_ms"] = decode_ms(p, stack, xd, posd, seqs, kr, lens, outs, args, torch, dev)
        if timing:
            # per-class launch durations of one eager forward (HIP events on the stream)
            for c in range(len(zsa.KCLASS_NAMES)):
                zsa.timing_arm(c, 1024)
            stack.forward(xd, posd, seqs, p.prune_after, kr, out=outs)
            torch.cuda.synchronize()
            cls = {}
            for c, name in enumerate(zsa.KCLASS_NAMES):
                n, t = zsa.timing_read(c)
                cls[name] = {"launches": n, "ms": t}
            rows_in, rows_after = layer_rows(p, plan)
            if (legs and p.dtype == "bf16" and p.d_model // p.n_heads in (64, 128)
                    and not args.forward_only and not args.no_backward):
                # the training step's backward (forward recomputed inside), as a graph
                g = torch.Generator().manual_seed(args.seed)
                dy = torch.randn(plan["final_rows"], p.d_model, generator=g).to(torch.bfloat16).to(dev)
                stack.backward(xd, posd, seqs, p.prune_after, kr, dy)
                r["backward_ms"] = graph_ms(
                    lambda: stack.backward(xd, posd, seqs, p.prune_after, kr, dy), args, torch)
            if legs and not args.forward_only and not args.no_backward:
                mouts = mstack.forward(xd, posd, seqs, p.prune_after, kr)
                r["mark_ms"] = graph_ms(
                    lambda: mstack.forward(xd, posd, seqs, p.prune_after, kr, out=mouts), args,
                    torch)
            r.update({"classes": cls, "gemm_flops": gemm_flops(p, rows_in, rows_after),
                      "rows": (rows_in, rows_after),
                      "work": class_work(p, lens, plan, rows_in, rows_after)})
        results[rate] = r
        if not args.no_graph:
            del g
    return lens, ws_np, x_np, results


def ceilings(torch, dev):
    """What this GPU sustains: a 1 GiB device-to-device copy (read + write
    bytes over time) and a large bf16 product through the vendor library
    (hipBLASLt), for reading the rooflines beside the published peaks."""
    out = {}
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(2):
        dst.copy_(src)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    out["hbm_copy_GBs"] = round(2.0 * n * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del src, dst
    m = 8192
    a = torch.randn(m, m, device=dev, dtype=torch.bfloat16)
    b = torch.randn(m, m, device=dev, dtype=torch.bfloat16)
    for _ in range(2):
        torch.matmul(a, b)
    e0.record()
    for _ in range(5):
        torch.matmul(a, b)
    e1.record()
    torch.cuda.synchronize()
    out["bf16_gemm_8192_hipblaslt_TFLOPs"] = round(2.0 * m ** 3 * 5 / (e0.elapsed_time(e1) * 1e-3)
                                                  / 1e12, 1)
    return out


def decode_ms(p, stack, xd, posd, seqs, kr, lens, outs, args, torch, dev):
    """Time of one generated row per sequence after the pruned prefill at
    this keep rate (the cache then holds each layer's kept rows), as a
    replayed HIP graph at a fixed cache length."""
    cap = max(lens) + 8
    cache = stack.kv_cache(seqs.batch, cap, dev)
    stack.forward(xd, posd, seqs, p.prune_after, kr, out=outs, kv_cache=cache)
    lens0 = stack.kv_lengths(seqs, p.prune_after, kr)
    g = torch.Generator().manual_seed(args.seed)
    x_new = torch.randn(seqs.batch, p.d_model, generator=g).to(torch.bfloat16).to(dev)
    y = stack.decode_step(x_new, lens, cache, lens0.copy())
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            stack.decode_step(x_new, lens, cache, lens0.copy(), out=y)
    torch.cuda.current_stream().wait_stream(s)
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / args.steps


def sweep_of(results, rates):
    base = results.get(1.0)
    out = []
    for rate in rates:
        r = results[rate]
        label = rate if rate != PER_SEQ else "per sequence, uniform in [0.05, 1]"
        out.append({"keep_rate": label, "tokens_per_s": round(r["tok_s"], 1),
                    "ms_per_step": round(r["ms"], 4),
                    "step_ms_median_p10_p90": [round(r["step_ms"][q], 4)
                                               for q in ("median", "p10", "p90")],
                    "speedup_vs_keep_rate_1": None if base is None else round(base["ms"] / r["ms"], 3),
                    "rows_after_last_prune": r["kept_rows_final"]})
        if "mark_ms" in r:
            # the same stack with rows marked instead of removed (Appendix B):
            # the ratio is the part of the speedup that compaction delivers
            out[-1]["mark_mode_ms_per_step"] = round(r["mark_ms"], 4)
            out[-1]["compaction_speedup_vs_mark_mode"] = round(r["mark_ms"] / r["ms"], 3)
        if "backward_ms" in r:
            out[-1]["backward_ms_per_step"] = round(r["backward_ms"], 4)
            out[-1]["train_step_ms"] = round(r["ms"] + r["backward_ms"], 4)
        if "decode_ms" in r:
            out[-1]["decode_ms_per_step"] = round(r["decode_ms"], 4)
            out[-1]["ttft_ms"] = round(r["ms"] + r["decode_ms"], 4)
            if base is not None and "decode_ms" in base:
                out[-1]["ttft_speedup_vs_keep_rate_1"] = round(
                    (base["ms"] + base["decode_ms"]) / (r["ms"] + r["decode_ms"]), 3)
    return out


def describe(p):
    kind = "decoder (RMSNorm, SwiGLU, RoPE)" if p.kind == 1 else "pre-LN block (LayerNorm, GELU, biases)"
    mask = "causal" if p.causal else "bidirectional"
    if len(p.prune_after) == p.n_layers:
        where = "after every layer"
    else:
        where = "after layers " + "/".join(map(str, p.prune_after))
    heads = f"H{p.n_heads}" + (f"/KV{p.kv_heads}" if p.kv_heads != p.n_heads else "")
    last = ", last row always kept" if p.force_keep_last else ""
    rows = (f"{p.batch} sequences of U[{p.min_len}, {p.seq_len}] rows" if p.ragged
            else f"{p.batch}x{p.seq_len} rows")
    return (f"{p.name}: {p.n_layers}-layer {mask} {kind} d{p.d_model} {heads} FFN{p.d_ff}, "
            f"{rows}, pruned {where} (tau {p.tau}){last}")


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args)
        return
    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the pruned stack "
              f"is measured on a single MI355X and this build has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2509_01190_amd import workloads as W
    from paper_2509_01190_amd import zsa

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        src = torch.empty(args.copy_calibration, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.copy_calibration}))
        return
    if args.gemm_table:
        gemm_table(args, torch, W, zsa, dev)
        return
    p = W.PRESETS[args.workload]
    rates = [float(r) for r in args.keep_rates.split(",")] if args.keep_rates else list(p.keep_rates)
    if HEADLINE_RATE not in rates:
        rates.append(HEADLINE_RATE)
    if 1.0 in rates:      # keep rate 1 first: the reference of the speedups
        rates = [1.0] + [r for r in rates if r != 1.0]
    lens, ws_np, x_np, results = measure(p, rates, args, torch, W, zsa, dev, timing=True, legs=True)
    sweep = sweep_of(results, rates)
    roofline = projection_roofline(p, results, rates, measured_traffic(p.name), zsa)
    head = results[HEADLINE_RATE]
    phases = {name: round(v["ms"], 4) for name, v in head["classes"].items() if v["launches"]}
    per_class = class_rooflines(p, head)

    cpu_budget = args.cpu_seconds
    others = {}
    legs = set(w for w in args.legs.split(",") if w)
    for name in [w for w in args.also.split(",") if w and w != p.name]:
        q = W.PRESETS[name]
        # keep rate 1 first, the reference of the speedups
        q_rates = [1.0] + [r for r in q.keep_rates if r != 1.0]
        if q.per_seq_rates:
            q_rates.append(PER_SEQ)
        q_lens, q_ws, q_x, res = measure(q, q_rates, args, torch, W, zsa, dev, timing=True,
                                         legs=name in legs)
        others[name] = {"workload": describe(q), "sweep": sweep_of(res, q_rates),
                        "roofline": projection_roofline(q, res, q_rates, None, zsa)}
        if cpu_budget > 0 and name in CPU_SAMPLES:
            # the oracle on a bounded sample of this workload (its keep rate
            # 0.5, or the per-sequence rates)
            q_rate = PER_SEQ if q.per_seq_rates else 0.5
            kr = W.keep_rates(q, args.seed, None if q_rate == PER_SEQ else q_rate)
            seqs, runs = CPU_SAMPLES[name](q_lens)
            others[name]["cpu_baseline"] = cpu_baseline(q, q_ws, q_x, q_lens, kr, seqs, runs,
                                                        cpu_budget)
        del q_ws, q_x

    ceil = ceilings(torch, dev)

    cpu = None
    if cpu_budget > 0:
        kr = W.keep_rates(p, args.seed, HEADLINE_RATE)
        cpu = cpu_baseline(p, ws_np, x_np, lens, kr, [0], 3, cpu_budget)

    line = {
        "metric": METRIC, "value": round(head["tok_s"], 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(head["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": p.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) hidden rows)",
        "config": {"workload": describe(p),
                   "keep_rate": HEADLINE_RATE, "global_batch": p.batch, "seq_len": p.seq_len,
                   "graph": not args.no_graph, "seed": args.seed},
        "step_ms_median_p10_p90": [round(head["step_ms"][q], 4) for q in ("median", "p10", "p90")],
        "sweep": sweep, "phases_ms_at_headline": phases, "roofline": roofline,
        "roofline_by_class_at_headline": per_class, "measured_ceilings": ceil,
        "other_workloads": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


# CPU-oracle samples of the other workloads: (sequences, runs) from the lengths
CPU_SAMPLES = {
    "bert": lambda lens: ([0, 1, 2, 3], 3),
    "tiny": lambda lens: (list(range(len(lens))), 3),
    "dec7b": lambda lens: ([0], 1),
    # the shortest and the longest sequence of the ragged batch
    "ragged": lambda lens: ([int(np.argmin(lens)), int(np.argmax(lens))], 1),
}


def projection_roofline(p, results, rates, traffic, zsa):
    """The projections of one workload over its sweep against the bf16 MFMA
    peak: algorithmic FLOPs over the summed event-timed launch durations."""
    g_ms = sum(results[r]["classes"]["gemm"]["ms"] for r in rates)
    g_n = sum(results[r]["classes"]["gemm"]["launches"] for r in rates)
    n_proj = 4 * p.n_layers * len(rates)      # QKV, output, up, down per layer
    g_flops = sum(results[r]["gemm_flops"] for r in rates)
    achieved = g_flops / (g_ms * 1e-3) / 1e12 if g_ms > 0 else 0.0
    # dominant kernel class over the whole sweep (every rate runs the same
    # number of steps, so this is also the mix a profiler sees)
    tot = {name: sum(results[r]["classes"][name]["ms"] for r in rates) for name in zsa.KCLASS_NAMES}
    return {"kernel": "projections (gemm_bf16_* or gemm_skinny_kernel, plus splitk_reduce_kernel "
                      "where K is split)",
            "bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": None if traffic is None else round(traffic),
            "traffic_unit": "HBM bytes per projection (FETCH_SIZE + WRITE_SIZE, copy-scaled)",
            "algorithmic_bytes_per_projection": round(gemm_bytes(p, results, rates) / n_proj),
            "algorithmic_flops_per_projection": round(g_flops / n_proj),
            "avg_us_per_projection": round(g_ms * 1e3 / n_proj, 2), "projections": n_proj,
            "launches": g_n, "dominant_class": max(tot, key=tot.get),
            "class_share_of_gpu_time": {k: round(v / max(sum(tot.values()), 1e-12), 4)
                                        for k, v in tot.items() if v > 0}}


def class_rooflines(p, head):
    """Every kernel class at one keep rate against its own bound."""
    per_class = {"gemm": {"bound": "mfma", "achieved": round(
        head["gemm_flops"] / (head["classes"]["gemm"]["ms"] * 1e-3) / 1e12, 1), "unit": "TFLOP/s",
        "peak": PEAK_BF16_TFLOPS}}
    for name, (unit, amount) in head["work"].items():
        t = head["classes"][name]["ms"] * 1e-3
        if t <= 0:
            continue
        if unit == "TFLOP/s":
            ach, peak, bound = amount / t / 1e12, PEAK_BF16_TFLOPS, "mfma"
        else:
            ach, peak, bound = amount / t / 1e9, PEAK_HBM_GBS, "hbm"
        per_class[name] = {"bound": bound, "achieved": round(ach, 1), "unit": unit,
                           "peak": peak}
    for v in per_class.values():
        v["frac"] = round(v["achieved"] / v["peak"], 4)
    # attention and the score sweep take one exp per (query, key, head) pair:
    # their second bound is the exp rate
    hd = p.d_model // p.n_heads
    for name, flop_per_exp in (("attention", 4 * hd), ("score", 2 * hd)):
        if name in per_class:
            t = head["classes"][name]["ms"] * 1e-3
            rate = head["work"][name][1] / flop_per_exp / t
            per_class[name]["exp_bound"] = {"achieved_exp_per_s": float(f"{rate:.4g}"),
                                            "peak_exp_per_s": PEAK_EXP_PER_S,
                                            "frac": round(rate / PEAK_EXP_PER_S, 4)}
    return per_class


if __name__ == "__main__":
    main()
