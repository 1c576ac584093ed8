#!/usr/bin/env python3
"""Throughput of the pruned layer-stack forward on one MI355X.

Workload: a 12-layer BERT-base-shaped encoder (d = 768, 12 heads, FFN 3072,
exact GELU, pre-LN), 32 sequences x 512 rows, bf16 storage, random-init
N(0, 0.02) weights and N(0, 1) hidden rows (synthetic), pruned after
layers 3, 6 and 9. One step = one whole stack forward over the batch
(norms, projections, attention, contribution scores, top-k, compaction),
replayed as a HIP graph with every input already in HBM.

The keep rate is swept over 1.0, 0.7, 0.5, 0.3, 0.1; `value` is the
throughput at keep rate 0.5 (input tokens per second), the other points go
to `sweep` with their speedup over keep rate 1. `other_workloads` adds the
same sweep for the paper's own schedule (Eq. 2 after every layer, tau = 5)
on a GPT-2-small-shaped causal stack at 128, 512 and 1024 rows per sequence,
for a LLaMA-3-8B-shaped slice (with its decode step), and for the other
workloads of the method's scope: a 1B- and a 7B-shaped decoder prefill, a
ragged batch of one 7B-shaped layer with per-sequence keep rates, and the
tiny encoder the oracle runs in full.

`roofline` is reported for the kernel class with the largest share of GPU
time, the projections: algorithmic FLOPs (2 * rows * out * in per
projection) over the summed durations of the projection kernels (the GEMM
and, where K is split, its reduce), measured with HIP events on the launch
stream, against the 2.5 PFLOP/s dense bf16 MFMA peak; `traffic` is the
counter-measured HBM bytes per projection. `roofline_by_class_at_headline`
puts every kernel class against its own bound, and `measured_ceilings`
gives what the GPU sustains on a plain copy and a vendor bf16 GEMM.
`cpu_baseline` times the float64 CPU oracle on a bounded sample of the same
workload.
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
# exp throughput: v_exp_f32 is a quarter-rate VALU op, so a wave64 takes 16
# cycles: 256 CUs x 4 SIMDs x 4 exp per clock x 2.4 GHz
PEAK_EXP_PER_S = 256 * 4 * 4 * 2.4e9
HEADLINE_RATE = 0.5
# sweep key of presets whose keep rates are drawn per sequence
PER_SEQ = "per_sequence"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="bert")
    ap.add_argument("--keep-rates", default=None, help="comma-separated sweep")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--also", default="gpt2,gpt2_n128,gpt2_n1024,llama3_8b,dec1b,dec7b,ragged,tiny",
                    help="comma-separated presets whose keep-rate sweeps are reported beside "
                         "the headline workload")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches instead")
    ap.add_argument("--forward-only", action="store_true",
                    help="skip the decode, backward and mark-mode legs (counter runs of the forward)")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the backward and mark-mode legs (traces of the forward and decode)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target wall time of the CPU-oracle sample (0 disables it)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run one plain device copy of BYTES bytes (profiled under "
                         "rocprofv3 --pmc to scale FETCH_SIZE / WRITE_SIZE) and exit")
    ap.add_argument("--summarize-pmc", nargs=4, default=None,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="turn rocprofv3 --pmc counter CSVs of this bench and of the copy "
                         "calibration into " + "profiles/gemm_traffic.json and exit")
    ap.add_argument("--copy-bytes", type=int, default=256 << 20)
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


def measured_traffic():
    """HBM bytes per projection from the committed counter summary, or None
    when the GEMM source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != gemm_source_hash():
        return None
    return t.get("hbm_bytes_per_projection")


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
            score_flops += sum(2.0 * n * n * hd * H * frac for n in cur)
            point += 1
            cur = counts[point]
    gather_bytes = 0.0
    select_bytes = 0.0
    for pt in range(len(p.prune_after)):
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


def cpu_baseline(p, ws_np, x_np, lens, rate, budget_s):
    """The float64 oracle (as it stands) on a bounded sample of sequences."""
    from oracle import zsa_oracle as O
    from paper_2509_01190_amd import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    ocfg = O.LayerCfg(p.kind, p.d_model, p.n_heads, p.d_ff, p.causal, p.norm_eps, p.rope_theta,
                      p.tau)
    ows = [{k: (None if v is None else W.as_f64(W.to_storage(v, p.dtype))) for k, v in w.items()}
           for w in ws_np]
    x64 = W.as_f64(W.to_storage(x_np, p.dtype))
    cu = W.cu_seqlens(lens)
    done_rows, elapsed, nseq = 0, 0.0, 0
    while nseq < len(lens) and (elapsed < budget_s * 0.5 or nseq == 0):
        b = nseq
        n = lens[b]
        xb = x64[cu[b]:cu[b + 1]]
        t0 = time.perf_counter()
        O.stack_forward(xb, np.arange(n), [0, n], ows, ocfg, p.prune_after, [rate])
        elapsed += time.perf_counter() - t0
        done_rows += n
        nseq += 1
        per = elapsed / nseq
        if elapsed + per > budget_s:
            break
    return {"value": done_rows / elapsed, "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{nseq} of {len(lens)} sequences x {lens[0]} rows, keep_rate {rate}, "
                      f"float64 exact mode, {elapsed:.1f} s"}


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


def measure(p, rates, args, torch, W, zsa, dev, timing):
    """Graph-replayed step time of preset ``p`` at every keep rate (and, with
    ``timing``, per-class launch durations of one eager forward and the same
    stack in mark-only mode, rows marked instead of removed)."""
    lens = W.lengths(p, args.seed)
    ws_np = W.stack_weights(p, args.seed)
    x_np = W.hidden(p, args.seed, lens)
    dws = [{k: (None if v is None else W.to_storage(v, p.dtype).to(dev)) for k, v in w.items()}
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
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        plan = stack.plan(seqs, p.prune_after, kr)
        r = {"ms": ms, "tok_s": tokens / (ms * 1e-3), "kept_rows_final": plan["final_rows"]}
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
            if (p.dtype == "bf16" and p.d_model // p.n_heads in (64, 128) and not args.forward_only
                    and not args.no_backward):
                # the training step's backward (forward recomputed inside), as a graph
                g = torch.Generator().manual_seed(args.seed)
                dy = torch.randn(plan["final_rows"], p.d_model, generator=g).to(torch.bfloat16).to(dev)
                stack.backward(xd, posd, seqs, p.prune_after, kr, dy)
                r["backward_ms"] = graph_ms(
                    lambda: stack.backward(xd, posd, seqs, p.prune_after, kr, dy), args, torch)
            if not args.forward_only and not args.no_backward:
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
    p = W.PRESETS[args.workload]
    rates = [float(r) for r in args.keep_rates.split(",")] if args.keep_rates else list(p.keep_rates)
    if HEADLINE_RATE not in rates:
        rates.append(HEADLINE_RATE)
    lens, ws_np, x_np, results = measure(p, rates, args, torch, W, zsa, dev, timing=True)
    sweep = sweep_of(results, rates)

    # dominant kernel class over the whole sweep (every rate runs the same
    # number of steps, so this is also the mix a profiler sees)
    tot = {name: sum(results[r]["classes"][name]["ms"] for r in rates) for name in zsa.KCLASS_NAMES}
    dom = max(tot, key=tot.get)
    g_ms = sum(results[r]["classes"]["gemm"]["ms"] for r in rates)
    g_n = sum(results[r]["classes"]["gemm"]["launches"] for r in rates)
    n_proj = 4 * p.n_layers * len(rates)      # QKV, output, up, down per layer
    g_flops = sum(results[r]["gemm_flops"] for r in rates)
    achieved = g_flops / (g_ms * 1e-3) / 1e12 if g_ms > 0 else 0.0
    traffic = measured_traffic()
    roofline = {"kernel": "projections (gemm_bf16_* or gemm_skinny_kernel, plus splitk_reduce_kernel where K is split)",
                "bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None if traffic is None else round(traffic),
                "traffic_unit": "HBM bytes per projection (FETCH_SIZE + WRITE_SIZE, copy-scaled)",
                "algorithmic_bytes_per_projection": round(gemm_bytes(p, results, rates) / n_proj),
                "avg_us_per_projection": round(g_ms * 1e3 / n_proj, 2), "projections": n_proj,
                "launches": g_n, "dominant_class": dom}
    head = results[HEADLINE_RATE]
    phases = {name: round(v["ms"], 4) for name, v in head["classes"].items() if v["launches"]}
    # every kernel class against its own roofline, at the headline keep rate
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

    # the paper's every-layer schedule on a GPT-2-small-shaped causal stack
    others = {}
    for name in [w for w in args.also.split(",") if w and w != p.name]:
        q = W.PRESETS[name]
        # keep rate 1 first, the reference of the speedups
        rates = [1.0] + [r for r in q.keep_rates if r != 1.0]
        if q.per_seq_rates:
            rates.append(PER_SEQ)
        _, _, _, res = measure(q, rates, args, torch, W, zsa, dev, timing=False)
        others[name] = {"workload": describe(q), "sweep": sweep_of(res, rates)}

    ceil = ceilings(torch, dev)

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(p, ws_np, x_np, lens, HEADLINE_RATE, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": round(head["tok_s"], 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(head["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": p.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) hidden rows)",
        "config": {"workload": describe(p),
                   "keep_rate": HEADLINE_RATE, "global_batch": p.batch, "seq_len": p.seq_len,
                   "graph": not args.no_graph},
        "sweep": sweep, "phases_ms_at_headline": phases, "roofline": roofline,
        "roofline_by_class_at_headline": per_class, "measured_ceilings": ceil,
        "other_workloads": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
