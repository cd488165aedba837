"""Benchmark of the ProxyAttn prefill hot path on one MI355X.

One step = the whole path on one synthetic layer already resident in HBM:
proxyattn_estimate -> proxyattn_select_budget -> proxyattn_prepare_kv ->
proxyattn_block_sparse_prefill_blocked.  The dense baseline runs the same
attention kernel over every causal block on the step's K/V copy; its time
includes one copy as well.
Default workload: Llama-3-8B-shaped attention layer at 131072 tokens (32 query
/ 8 KV heads, d 128, block 128, 4 proxy groups, stride 4, gamma 0.95, head
deviation 0.3), bf16.

Prints ONE JSON line (rank 0).  Besides the step time it reports the stage
times, the same-build dense kernel's time, dense-equivalent TFLOP/s, the
estimation overhead, sparsity, a roofline entry for the dominant kernel
(block-sparse attention, MFMA-bound) and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse prefill attention ms + dense-equiv TFLOP/s at 128K; estimation overhead %"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3_8b_n131072")
    ap.add_argument("--gamma", type=float, default=None)
    ap.add_argument("--noise", type=float, default=None, help="head deviation sigma")
    ap.add_argument("--num-proxy-groups", type=int, default=None)
    ap.add_argument("--min-budget", type=int, default=None)
    ap.add_argument("--seq-len", type=int, default=None,
                    help="override the workload's sequence length (same recipe and seed)")
    ap.add_argument("--dense-steps", type=int, default=3)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-rows", type=int, default=24,
                    help="block rows of the oracle sample (all heads)")
    ap.add_argument("--sweep", choices=sorted(SWEEPS), default=None,
                    help="print one JSON line per point of a workload sweep instead")
    ap.add_argument("--work-orders", action="store_true",
                    help="time the sparse attention call of --workload under each work-item "
                         "order (one JSON line per order) instead")
    ap.add_argument("--stack", type=int, default=None, metavar="LAYERS",
                    help="time a stack of LAYERS layers of --workload (layer l drawn with seed l; "
                         "one JSON line per layer, then the totals)")
    ap.add_argument("--ttft", action="store_true",
                    help="with --stack: run a LAYERS-layer decoder prefill around the path "
                         "(projections, RoPE, MLP; one timed region) and report the "
                         "time-to-first-token with the sparse path vs the dense kernel")
    ap.add_argument("--shard", type=int, default=None, metavar="P",
                    help="time --workload with one proxy group per KV head, whole and in P "
                         "head shards (each as one of P GPUs would run it); one JSON line")
    ap.add_argument("--stack-workers", type=int, default=4,
                    help="processes generating stack layers ahead of the GPU")
    ap.add_argument("--profile-summary", metavar="DIR", default=None,
                    help="summarise the rocprofv3 runs under DIR (no GPU): write "
                         "profiles/attn_traffic.json and print a markdown summary")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (scales the FETCH_SIZE / "
                         "WRITE_SIZE counters) and exit")
    return ap.parse_args()


def cpu_baseline(wl, q, k, v, sample_rows: int):
    """Time the oracle on a bounded sample and scale it to one full step.

    Sample: the last-block masses and budgets in full (they are per head and
    small), plus proxy scores, lists and attention for `sample_rows` seeded
    block rows (all heads).  Per-row costs grow linearly with the row index,
    so the sampled rows' time is scaled by sum(m+1 over all rows) / sum(m+1
    over the sample).
    """
    from threadpoolctl import threadpool_info
    from oracle import proxyattn_oracle as O
    mq = wl.num_blocks
    rng = np.random.default_rng(12345)
    rows = np.sort(rng.choice(mq, size=min(sample_rows, mq), replace=False))
    sc = O.default_scale(wl.head_dim)
    t0 = time.perf_counter()
    qg, kg = O.pool_proxy_heads(q, k, wl.num_proxy_groups, wl.stride, wl.dtype)
    t1 = time.perf_counter()
    logA, _ = O.proxy_block_logscore(qg, kg, wl.seq_len, wl.block_size, wl.stride, sc, rows=rows)
    t2 = time.perf_counter()
    mass = O.lastblock_mass(q, k, wl.block_size, sc)
    counts, _ = O.budget_counts(mass, wl.gamma, wl.min_budget_tokens, wl.block_size)
    t3 = time.perf_counter()
    bc, bi = O.select_blocks(logA, counts, wl.num_q_heads, rows=rows)
    t4 = time.perf_counter()
    qrows = np.concatenate([np.arange(m * wl.block_size, min((m + 1) * wl.block_size, wl.seq_len))
                            for m in rows])
    O.block_sparse_attention(q, k, v, bc, bi, wl.block_size, sc, query_rows=qrows)
    t5 = time.perf_counter()
    weight_all = mq * (mq + 1) / 2
    weight_s = float(np.sum(rows + 1))
    scale_rows = weight_all / weight_s
    full_s = (t1 - t0) + (t3 - t2) + ((t2 - t1) + (t4 - t3) + (t5 - t4)) * scale_rows
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as fh:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")),
                             None)
    except OSError:
        pass
    return {
        "value": round(full_s * 1e3, 1), "unit": "ms", "cores": int(threads), "kind": "oracle",
        "cpu_model": cpu_model, "host_cpus": os.cpu_count(),
        "sample": (f"pooling, last-block masses and budgets in full; proxy scores, lists and "
                   f"attention for {len(rows)} of {mq} block rows (all heads), scaled by causal "
                   f"work; measured {t5 - t0:.1f} s"),
    }


# sources the attention kernel is compiled from
KERNEL_SOURCES = ("attention.hip", "work_order.h", "common.h", "internal.h")
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "attn_traffic.json")


def kernel_sources_sha256() -> str:
    """Hash of the attention kernel's sources with // comments and
    whitespace removed, so that only a change to the code itself marks the
    committed traffic counters as stale."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2509_24745_amd", "csrc", f), encoding="utf-8") as fh:
            code = re.sub(r"//[^\n]*", "", fh.read())
        h.update(re.sub(r"\s+", "", code).encode())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per sparse attention launch from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE runs (copy-calibrated), or None when the kernel
    sources have changed since they were taken."""
    try:
        rec = json.load(open(TRAFFIC_JSON))
        sha = kernel_sources_sha256()
    except OSError:
        return None
    if rec.get("kernel_sources_sha256") != sha:
        return None
    return rec["fetch_bytes"] + rec["write_bytes"]


# The rocprofv3 runs --profile-summary reads (DIR = their output folder).
PROFILE_COMMANDS = [
    "rocprofv3 --kernel-trace --stats -T -f csv -d DIR/trace -o run -- "
    "python3 bench.py --steps 5 --warmup 2 --no-cpu-baseline",
    "rocprofv3 --pmc FETCH_SIZE -T -f csv --kernel-include-regex attn_kernel -d DIR/pmc_FETCH_SIZE "
    "-o run -- python3 bench.py --steps 1 --warmup 0 --no-dense --no-cpu-baseline",
    "rocprofv3 --pmc WRITE_SIZE -T -f csv --kernel-include-regex attn_kernel -d DIR/pmc_WRITE_SIZE "
    "-o run -- python3 bench.py --steps 1 --warmup 0 --no-dense --no-cpu-baseline",
    "rocprofv3 --pmc FETCH_SIZE -T -f csv -d DIR/cal_FETCH_SIZE -o run -- "
    "python3 bench.py --calibrate-copy",
    "rocprofv3 --pmc WRITE_SIZE -T -f csv -d DIR/cal_WRITE_SIZE -o run -- "
    "python3 bench.py --calibrate-copy",
]


def _kernel_label(name: str) -> str:
    import re
    m = re.match(r"_ZN2pa\d+(\w+?)I(DF16b|f)Li(\d+)E(?:Li(\d+)E)?(?:Lb([01])E)?", name)
    if not m:
        m2 = re.match(r"_ZN2pa\d+(\w+?)ILi(\d+)EE", name)   # one integer parameter
        if m2:
            return f"{m2.group(1)}<{m2.group(2)}>"
        return name.split("(")[0][:48]
    kind, t, a, b, flag = m.groups()
    t = "bf16" if t == "DF16b" else "f32"
    if kind == "attn_kernel":
        return f"attn_kernel<{t},d{a},b{b},{'dense' if flag == '1' else 'sparse'}>"
    if kind == "est_rowmax_kernel":
        return f"est_rowmax_kernel<{t},d{a},b'{b}>"
    return f"{kind}<{t},{a}>" if b is None else f"{kind}<{t},{a},{b}>"


def profile_summary(d: str, workload: str) -> str:
    """Summarise rocprofv3 output under `d` (the PROFILE_COMMANDS runs): write
    profiles/attn_traffic.json and return a markdown summary."""
    import csv
    import glob

    def rows(sub, pattern):
        files = glob.glob(os.path.join(d, sub, pattern))
        if not files:
            raise SystemExit(f"no {pattern} under {os.path.join(d, sub)}")
        with open(files[0]) as fh:
            return list(csv.DictReader(fh))

    def counter(sub, name, kernel_pred):
        vals = [float(r["Counter_Value"]) for r in rows(sub, "*counter_collection.csv")
                if r["Counter_Name"] == name and kernel_pred(r["Kernel_Name"])]
        if not vals:
            raise SystemExit(f"no {name} values in {sub}")
        return sum(vals) / len(vals), len(vals)

    sparse = lambda k: "attn_kernel" in k and "Lb0E" in k
    copy = lambda k: "copy" in k.lower()
    f_kib, nf = counter("pmc_FETCH_SIZE", "FETCH_SIZE", sparse)
    w_kib, nw = counter("pmc_WRITE_SIZE", "WRITE_SIZE", sparse)
    cf_kib, _ = counter("cal_FETCH_SIZE", "FETCH_SIZE", copy)
    cw_kib, _ = counter("cal_WRITE_SIZE", "WRITE_SIZE", copy)
    gib_kib = float(1 << 20)               # a 1 GiB copy reads and writes 2^20 KiB
    f_scale, w_scale = gib_kib / cf_kib, gib_kib / cw_kib
    fetch_b, write_b = f_kib * 1024 * f_scale, w_kib * 1024 * w_scale
    rec = {"kernel": "attn_kernel<bf16,128,128,sparse>", "workload": workload,
           "kernel_sources_sha256": kernel_sources_sha256(),
           "fetch_bytes": fetch_b, "write_bytes": write_b, "fetch_kib": f_kib, "write_kib": w_kib,
           "copy_fetch_kib_per_gib": cf_kib, "copy_write_kib_per_gib": cw_kib}
    with open(TRAFFIC_JSON, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    stats = rows("trace", "*kernel_stats.csv")
    out = ["## Kernel trace (rocprofv3 --kernel-trace --stats)", "",
           "| kernel | calls | avg ms | min ms | max ms | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats:
        out.append(f"| {_kernel_label(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e6:.3f} | "
                   f"{float(r['MinNs']) / 1e6:.3f} | {float(r['MaxNs']) / 1e6:.3f} | "
                   f"{float(r['Percentage']):.2f} |")
    out += ["", "## HBM traffic of one sparse attention launch (rocprofv3 --pmc)", "",
            "| counter | attn_kernel (KiB, mean of %d / %d launches) | 1 GiB copy (KiB) | scale | bytes per launch |" % (nf, nw),
            "|---|---|---|---|---|",
            f"| FETCH_SIZE | {f_kib:.0f} | {cf_kib:.1f} | {f_scale:.4f} | {fetch_b:.4e} |",
            f"| WRITE_SIZE | {w_kib:.0f} | {cw_kib:.1f} | {w_scale:.4f} | {write_b:.4e} |",
            "", f"Traffic per launch: {fetch_b + write_b:.4e} bytes.", "",
            "Commands (repository root, one MI355X; DIR = the output folder):", ""]
    out += ["    " + c for c in PROFILE_COMMANDS]
    out += ["    python3 bench.py --profile-summary DIR"]
    return "\n".join(out) + "\n"


def vendor_dense_ms(wl, inputs, reps: int = 2):
    """torch's scaled_dot_product_attention restricted to its flash backend
    (AOTriton on ROCm; no fallback to the quadratic-memory math path) on the
    same Q/K/V, KV heads repeated for GQA: the vendor dense attention, for
    context.  None if that backend is unavailable."""
    import torch
    from torch.nn.attention import SDPBackend, sdpa_kernel
    q, k, v = inputs
    rep = wl.num_q_heads // wl.num_kv_heads
    qh = q.permute(1, 0, 2).unsqueeze(0).contiguous()
    kh = k.permute(1, 0, 2).repeat_interleave(rep, dim=0).unsqueeze(0).contiguous()
    vh = v.permute(1, 0, 2).repeat_interleave(rep, dim=0).unsqueeze(0).contiguous()
    try:
        with sdpa_kernel(SDPBackend.FLASH_ATTENTION):
            f = lambda: torch.nn.functional.scaled_dot_product_attention(qh, kh, vh, is_causal=True)
            f()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                f()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps
    except RuntimeError:
        return None
    finally:
        del qh, kh, vh


def measure(wl, steps: int, warmup: int, dense_steps: int, with_dense: bool = True,
            inputs=None, variant: str = "dynamic", static_k: int | None = None,
            dense_lse=None):
    """Time `steps` whole-path steps of workload `wl` (inputs resident in HBM).

    `variant` selects the budget step (Alg. 1 and Eq. 3):
      "dynamic"    proxyattn_select_budget (per-head budgets, constant reading);
      "row_ratio"  proxyattn_budget + proxyattn_select_topk, per-row-ratio reading;
      "static"     one budget of `static_k` blocks for every head
                   (proxyattn_select_topk, constant reading; no budget step).
    Returns (results, host arrays or None, device inputs).  With a dense
    reference (`with_dense`, or `dense_lse` passed in) the results include
    the attention-mass recall of the sparse lists, exp(lse_sparse - lse_dense)
    per (head, row).
    """
    import torch
    from paper_2509_24745_amd import proxyattn as pa
    from paper_2509_24745_amd.synth import generate

    prob = pa.Problem(seq_len=wl.seq_len, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                      head_dim=wl.head_dim, block_size=wl.block_size,
                      num_proxy_groups=wl.num_proxy_groups, stride=wl.stride, dtype=wl.dtype)
    host = None
    if inputs is None:
        print(f"[bench] generating {wl.name} N={wl.seq_len} gamma={wl.gamma} "
              f"sigma={wl.structure.noise} G={wl.num_proxy_groups}", file=sys.stderr, flush=True)
        t = time.time()
        host = generate(wl)
        print(f"[bench] generated in {time.time() - t:.1f}s", file=sys.stderr, flush=True)
        dt = prob.torch_dtype
        inputs = tuple(torch.from_numpy(host[x]).to(dt).cuda() for x in ("q", "k", "v"))
    q, k, v = inputs
    want_q = (wl.seq_len, wl.num_q_heads, wl.head_dim)
    want_kv = (wl.seq_len, wl.num_kv_heads, wl.head_dim)
    if tuple(q.shape) != want_q or tuple(k.shape) != want_kv or tuple(v.shape) != want_kv:
        raise ValueError(f"inputs {tuple(q.shape)}/{tuple(k.shape)} do not match {wl.name}")
    bufs = pa.Buffers(prob)
    stream = torch.cuda.current_stream()
    if variant == "static":
        bufs.head_count.fill_(int(static_k))
        torch.cuda.synchronize()
    elif variant not in ("dynamic", "row_ratio"):
        raise ValueError(f"unknown variant {variant}")

    def select(st):
        if variant == "dynamic":
            pa.proxyattn_select_budget(prob, bufs.logscore, bufs.mass, wl.gamma,
                                       wl.min_budget_tokens, bufs.head_count, bufs.block_count,
                                       bufs.block_index, st)
            return
        if variant == "row_ratio":
            pa.proxyattn_budget(prob, bufs.mass, wl.gamma, wl.min_budget_tokens, bufs.head_count,
                                st)
        mode = pa.TOPK_ROW_RATIO if variant == "row_ratio" else pa.TOPK_CONSTANT
        pa.proxyattn_select_topk(prob, bufs.logscore, bufs.head_count, mode, bufs.block_count,
                                 bufs.block_index, st)

    # the K/V copy the attention kernels read: made once per step from the
    # layer's K and V (proxyattn_prepare_kv), then read by the sparse call
    # and, outside the step, by the dense baseline
    kvb = torch.empty(pa.proxyattn_kv_blocked_size(prob), dtype=torch.uint8, device="cuda")
    qws = torch.empty(pa.proxyattn_blocked_workspace_size(prob), dtype=torch.uint8, device="cuda")

    def step(ev=None, st=None):
        st = stream if st is None else st
        if ev: ev[0].record(st)
        pa.proxyattn_estimate(prob, q, k, bufs.logscore, bufs.mass, bufs.workspace, st)
        if ev: ev[1].record(st)
        select(st)
        if ev: ev[2].record(st)
        pa.proxyattn_prepare_kv(prob, k, v, kvb, st)
        if ev: ev[3].record(st)
        pa.proxyattn_block_sparse_prefill_blocked(prob, q, kvb, bufs.block_count,
                                                  bufs.block_index, bufs.out, bufs.lse, qws, st)
        if ev: ev[4].record(st)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    # whole steps as one region with no event inside it (an event record
    # costs a few microseconds of GPU time, a visible share of a short
    # sequence's step) ...
    start.record(stream)
    for i in range(steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop) / steps
    # ... then the same steps with an event between stages, for the breakdown
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    t_est = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    t_sel = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    t_prep = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    t_attn = float(np.mean([e[3].elapsed_time(e[4]) for e in evs]))
    per_step = [e[0].elapsed_time(e[4]) for e in evs]   # estimate start to attention end
    # estimation + selection as a share of the stage-timed step (both sides
    # carry the same event overhead)
    est_share = (t_est + t_sel) / (t_est + t_sel + t_prep + t_attn)
    print(f"[bench] {wl.name}: {ms_total:.3f} ms/step (est {t_est:.3f}, sel {t_sel:.3f}, "
          f"prep {t_prep:.3f}, attn {t_attn:.3f})", file=sys.stderr, flush=True)

    mq, hq, d, b, n = prob.num_blocks, prob.num_q_heads, prob.head_dim, prob.block_size, prob.seq_len
    total_blocks = int(bufs.block_count.sum().item())
    counts = bufs.head_count.cpu().numpy()
    causal_blocks = hq * mq * (mq + 1) // 2
    f_dense = 4.0 * hq * d * n * (n + 1) / 2          # dense-equivalent causal flops
    f_attn = 4.0 * b * b * d * total_blocks            # flops the sparse kernel computes
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    achieved = f_attn / (t_attn * 1e-3) / 1e12
    # the same step captured once in a HIP graph and replayed (no host launch work)
    t_graph = None
    ref_count = bufs.block_count.clone()
    if steps > 0:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step(st=side)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(st=torch.cuda.current_stream())   # the capture stream
        graph.replay()
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(steps):
            graph.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        t_graph = g0.elapsed_time(g1) / steps
        # a replay must reproduce the eager step (same buffers, deterministic kernels)
        if not torch.equal(bufs.block_count, ref_count):
            raise RuntimeError("graph replay differs from the eager step")
        del graph
    t_dense = t_dense_attn = None
    if with_dense:
        # the dense kernel on the K/V copy of the last step; its time adds the
        # copy's, so that both sides include one proxyattn_prepare_kv
        de = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        dense_out = torch.empty_like(bufs.out)
        pa.proxyattn_dense_prefill_blocked(prob, q, kvb, dense_out, None, qws, stream)
        torch.cuda.synchronize()
        de[0].record(stream)
        for _ in range(dense_steps):
            pa.proxyattn_dense_prefill_blocked(prob, q, kvb, dense_out, None, qws, stream)
        de[1].record(stream)
        torch.cuda.synchronize()
        t_dense_attn = de[0].elapsed_time(de[1]) / dense_steps
        t_dense = t_prep + t_dense_attn
        print(f"[bench] dense {t_dense_attn:.3f} ms (+ prep {t_prep:.3f})", file=sys.stderr,
              flush=True)
        dense_lse = torch.empty_like(bufs.lse)
        pa.proxyattn_dense_prefill_blocked(prob, q, kvb, dense_out, dense_lse, qws, stream)
        torch.cuda.synchronize()
        del dense_out
    recall = None
    if dense_lse is not None:
        # share of each row's full causal attention mass inside its selected blocks
        rec = torch.exp(bufs.lse - dense_lse).clamp_(max=1.0)
        per_head = rec.mean(dim=1)
        recall = {"mean": float(rec.mean()), "worst_head_mean": float(per_head.min()),
                  "p01_row": float(torch.quantile(rec.flatten()[::97].float(), 0.01))}
    res = {
        "ms_total": ms_total, "t_est": t_est, "t_sel": t_sel, "t_attn": t_attn, "t_dense": t_dense,
        "step_median": float(np.median(per_step)) if per_step else None,
        "step_min": float(np.min(per_step)) if per_step else None,
        "sparsity": 1.0 - total_blocks / causal_blocks, "total_blocks": total_blocks,
        "f_dense": f_dense, "f_attn": f_attn, "achieved": achieved, "peak": peak,
        "head_count_min": int(counts.min()), "head_count_median": float(np.median(counts)),
        "head_count_max": int(counts.max()),
        "dense_mfma_frac": (4.0 * b * b * d * causal_blocks / (t_dense_attn * 1e-3) / 1e12 / peak)
        if t_dense_attn else None,
        "t_prep": t_prep, "t_dense_attn": t_dense_attn, "est_share": est_share,
        "variant": variant, "static_k": static_k, "recall": recall, "t_graph": t_graph,
        "head_count_mean": float(counts.mean()), "dense_lse": dense_lse,
    }
    return res, host, inputs


def summary_line(wl, r, steps):
    return {
        "workload": wl.name, "seq_len": wl.seq_len, "gamma": wl.gamma,
        "head_deviation": wl.structure.noise, "num_proxy_groups": wl.num_proxy_groups,
        "min_budget_tokens": wl.min_budget_tokens, "steps": steps,
        "ms_per_step": round(r["ms_total"], 4), "t_estimate_ms": round(r["t_est"], 4),
        "t_select_ms": round(r["t_sel"], 4), "t_prepare_kv_ms": round(r["t_prep"], 4),
        "t_attention_ms": round(r["t_attn"], 4),
        "t_dense_ms": round(r["t_dense"], 4) if r["t_dense"] else None,
        "speedup_vs_dense": round(r["t_dense"] / r["ms_total"], 3) if r["t_dense"] else None,
        "dense_equiv_tflops": round(r["f_dense"] / (r["ms_total"] * 1e-3) / 1e12, 2),
        "estimation_overhead_pct": round(100.0 * r["est_share"], 2),
        "sparsity": round(r["sparsity"], 4), "computed_blocks": r["total_blocks"],
        "attn_mfma_frac": round(r["achieved"] / r["peak"], 4),
        "dense_mfma_frac": round(r["dense_mfma_frac"], 4) if r["dense_mfma_frac"] else None,
        "head_count_min_median_max": [r["head_count_min"], r["head_count_median"],
                                      r["head_count_max"]],
        "stride": wl.stride, "variant": r["variant"], "static_k": r["static_k"],
        "recall": ({k: round(v, 5) for k, v in r["recall"].items()} if r["recall"] else None),
    }


DECODER_ALPHA = 0.125


class DecoderPrefill:
    """A Llama-3-8B-shaped decoder prefill in bf16 whose attention is the
    ProxyAttn path or, for the baseline, the dense kernel (the paper's
    end-to-end prefill setting, Sec. 4.3 and Fig. 1, with random weights).

    Layer l, on one stream:
        h = RMSNorm(x);  [q' | k' | v'] = h W_qkv;  RoPE on q' and k';
        Q = Qs + alpha q',  K = Ks + alpha k',  V = Vs + alpha v';
        o = attention(Q, K, V)          (estimate, select, prepare_kv and the
                                         sparse call, or prepare_kv and the
                                         dense call);
        x = x + o W_o;  [g | u] = RMSNorm(x) W_gu;  x = x + (SiLU(g) u) W_down.
    Qs, Ks, Vs are layer l's structured synthetic inputs.  Random weights on
    random hidden states give attention with no block structure, so the
    structure comes from the synthetic recipe and the projections are added
    to it: every attention reads what its layer's projections wrote, its
    output feeds the output projection, and each layer's hidden state is the
    next layer's input.  Weights are drawn per layer (about 0.44 GB a layer
    at the Llama-3-8B sizes), inputs and weights stay resident in HBM.
    """

    def __init__(self, wl, structured, hidden: int = 4096, inter: int = 14336,
                 alpha: float = DECODER_ALPHA, seed: int = 0, rope_theta: float = 500000.0):
        import torch
        from paper_2509_24745_amd import proxyattn as pa
        self.torch, self.pa, self.wl = torch, pa, wl
        self.hidden, self.inter, self.alpha = hidden, inter, alpha
        n, hq, hkv, d = wl.seq_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        self.n, self.hq, self.hkv, self.d = n, hq, hkv, d
        for qs, ks, vs in structured:
            if (tuple(qs.shape) != (n, hq, d) or tuple(ks.shape) != (n, hkv, d)
                    or tuple(vs.shape) != (n, hkv, d)):
                raise ValueError(f"structured inputs do not match {wl.name}")
        self.structured = structured
        self.layers = len(structured)
        self.prob = pa.Problem(seq_len=n, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                               block_size=wl.block_size, num_proxy_groups=wl.num_proxy_groups,
                               stride=wl.stride, dtype="bf16")
        self.bufs = pa.Buffers(self.prob)
        dev, bf = "cuda", torch.bfloat16
        self.kvb = torch.empty(pa.proxyattn_kv_blocked_size(self.prob), dtype=torch.uint8,
                               device=dev)
        self.qws = torch.empty(pa.proxyattn_blocked_workspace_size(self.prob), dtype=torch.uint8,
                               device=dev)
        self.q = torch.empty(n, hq, d, dtype=bf, device=dev)
        self.k = torch.empty(n, hkv, d, dtype=bf, device=dev)
        self.v = torch.empty(n, hkv, d, dtype=bf, device=dev)
        g = torch.Generator(device=dev).manual_seed(seed)

        def w(rows, cols):
            return torch.randn(rows, cols, device=dev, dtype=bf, generator=g) * rows ** -0.5

        self.weights = [(w(hidden, (hq + 2 * hkv) * d), w(hq * d, hidden), w(hidden, 2 * inter),
                         w(inter, hidden)) for _ in range(self.layers)]
        self.norm = [(torch.ones(hidden, device=dev, dtype=bf),
                      torch.ones(hidden, device=dev, dtype=bf)) for _ in range(self.layers)]
        inv = 1.0 / (rope_theta ** (torch.arange(0, d, 2, device=dev, dtype=torch.float32) / d))
        ang = torch.arange(n, device=dev, dtype=torch.float32)[:, None] * inv[None, :]
        self.cos = ang.cos().to(bf)[:, None, :]
        self.sin = ang.sin().to(bf)[:, None, :]

    def embed(self, seed: int = 1):
        """A seeded N(0, 1) hidden state [N, hidden] (the embedding output)."""
        g = self.torch.Generator(device="cuda").manual_seed(seed)
        return self.torch.randn(self.n, self.hidden, device="cuda", dtype=self.torch.bfloat16,
                                generator=g)

    def _rms(self, t, w):
        tf = t.float()
        return (tf * self.torch.rsqrt(tf.pow(2).mean(-1, keepdim=True) + 1e-5)).to(t.dtype) * w

    def _rope(self, t, heads):
        t = t.reshape(self.n, heads, self.d)
        h = self.d // 2
        a, b = t[..., :h], t[..., h:]
        return self.torch.cat((a * self.cos - b * self.sin, b * self.cos + a * self.sin), dim=-1)

    def attention(self, dense: bool, st):
        pa, prob, b, wl = self.pa, self.prob, self.bufs, self.wl
        if dense:
            pa.proxyattn_prepare_kv(prob, self.k, self.v, self.kvb, st)
            pa.proxyattn_dense_prefill_blocked(prob, self.q, self.kvb, b.out, b.lse, self.qws, st)
            return
        pa.proxyattn_estimate(prob, self.q, self.k, b.logscore, b.mass, b.workspace, st)
        pa.proxyattn_select_budget(prob, b.logscore, b.mass, wl.gamma, wl.min_budget_tokens,
                                   b.head_count, b.block_count, b.block_index, st)
        pa.proxyattn_prepare_kv(prob, self.k, self.v, self.kvb, st)
        pa.proxyattn_block_sparse_prefill_blocked(prob, self.q, self.kvb, b.block_count,
                                                  b.block_index, b.out, b.lse, self.qws, st)

    def layer(self, l: int, x, dense: bool, ev=None, hook=None):
        """Layer l on hidden state x (not modified); returns the next hidden state.
        `ev`: two events recorded around the attention; `hook(l)` runs right
        after the attention is enqueued (tests read the layer's buffers there)."""
        torch = self.torch
        n, hq, hkv, d, a = self.n, self.hq, self.hkv, self.d, self.alpha
        w_qkv, w_o, w_gu, w_dn = self.weights[l]
        n1, n2 = self.norm[l]
        qs, ks, vs = self.structured[l]
        st = torch.cuda.current_stream()
        qkv = self._rms(x, n1) @ w_qkv
        torch.add(qs, self._rope(qkv[:, :hq * d], hq), alpha=a, out=self.q)
        torch.add(ks, self._rope(qkv[:, hq * d:(hq + hkv) * d], hkv), alpha=a, out=self.k)
        torch.add(vs.view(n, hkv * d), qkv[:, (hq + hkv) * d:], alpha=a,
                  out=self.v.view(n, hkv * d))
        del qkv
        if ev:
            ev[0].record(st)
        self.attention(dense, st)
        if ev:
            ev[1].record(st)
        if hook:
            hook(l)
        x = x + self.bufs.out.view(n, hq * d) @ w_o
        gu = self._rms(x, n2) @ w_gu
        act = torch.nn.functional.silu(gu[:, :self.inter]) * gu[:, self.inter:]
        del gu
        return x + act @ w_dn

    def forward(self, x, dense: bool, timed: bool = False, hook=None):
        """All layers on the embedding output x; returns (hidden state, times).
        With `timed`, times = (total ms, attention ms summed over layers) from
        HIP events on the current stream, one region around all layers."""
        torch = self.torch
        st = torch.cuda.current_stream()
        evs = ([[torch.cuda.Event(enable_timing=True) for _ in range(2)]
                for _ in range(self.layers)] if timed else [None] * self.layers)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if timed:
            torch.cuda.synchronize()
            t0.record(st)
        for l in range(self.layers):
            x = self.layer(l, x, dense, evs[l], hook)
        if not timed:
            return x, None
        t1.record(st)
        torch.cuda.synchronize()
        return x, (t0.elapsed_time(t1), sum(e[0].elapsed_time(e[1]) for e in evs))


def _stack_layer(job):
    """Pool worker: draw layer `seed` of a stack and store its bf16 bits as .npy files."""
    wname, seed, outdir, threads = job
    from threadpoolctl import threadpool_limits
    from paper_2509_24745_amd.synth import WORKLOADS, generate, to_bf16_bits
    wl = WORKLOADS[wname].replace(seed=seed)
    with threadpool_limits(threads):
        g = generate(wl)
    paths = []
    for x in ("q", "k", "v"):
        path = os.path.join(outdir, f"layer{seed}_{x}.npy")
        np.save(path, to_bf16_bits(g.pop(x)))
        paths.append(path)
    return seed, paths


def _layer_stream(wname: str, layers: int, workers: int):
    """Yield (layer, (q, k, v) bf16 device tensors) for layers 0..layers-1 of
    workload `wname`, layer l drawn with seed l by `workers` spawned processes
    (started before this process touches the GPU), at most workers + 1 ahead
    of the consumer, and passed through .npy files."""
    import multiprocessing as mp
    import shutil
    import tempfile
    from paper_2509_24745_amd.synth import WORKLOADS
    base = WORKLOADS[wname]
    if base.dtype != "bf16":
        raise SystemExit("--stack runs bf16 workloads (layers pass as bf16 bits)")
    layer_bytes = 2 * base.seq_len * (base.num_q_heads + 2 * base.num_kv_heads) * base.head_dim
    tmp_root = None
    if os.path.isdir("/dev/shm"):
        st = os.statvfs("/dev/shm")
        if st.f_bavail * st.f_frsize > (workers + 2) * layer_bytes * 1.2:
            tmp_root = "/dev/shm"
    outdir = tempfile.mkdtemp(prefix="proxyattn_stack_", dir=tmp_root)
    threads = max(1, (os.cpu_count() or workers) // workers)
    pool = mp.get_context("spawn").Pool(workers)
    try:
        import torch
        pending = {}
        nxt = 0

        def fill():
            nonlocal nxt
            while nxt < layers and len(pending) < workers + 1:
                pending[nxt] = pool.apply_async(_stack_layer, ((wname, nxt, outdir, threads),))
                nxt += 1

        fill()
        for layer in range(layers):
            _, paths = pending.pop(layer).get()
            fill()
            bits = [np.load(p) for p in paths]
            for p in paths:
                os.remove(p)
            inputs = tuple(torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
                           for a in bits)
            del bits
            yield layer, inputs
    finally:
        pool.terminate()
        pool.join()
        shutil.rmtree(outdir, ignore_errors=True)


def run_stack(wname: str, layers: int, steps: int, warmup: int, dense_steps: int, workers: int):
    """The attention of a stack of `layers` layers of workload `wname`, layer
    l drawn with seed l: each layer timed like the default line (sparse path
    and dense kernel, one JSON line per layer), then the stack totals."""
    from paper_2509_24745_amd.synth import WORKLOADS
    base = WORKLOADS[wname]
    sums = {"t_total": 0.0, "t_est": 0.0, "t_sel": 0.0, "t_attn": 0.0, "t_dense": 0.0,
            "t_stages": 0.0, "blocks": 0,
            "causal": 0}
    for layer, inputs in _layer_stream(wname, layers, workers):
        wl = base.replace(seed=layer)
        res, _, _ = measure(wl, steps, warmup, dense_steps, with_dense=True, inputs=inputs)
        del inputs
        line = summary_line(wl, res, steps)
        line["layer"] = layer
        print(json.dumps(line), flush=True)
        sums["t_total"] += res["ms_total"]
        sums["t_est"] += res["t_est"]
        sums["t_sel"] += res["t_sel"]
        sums["t_attn"] += res["t_attn"]
        sums["t_stages"] += res["t_est"] + res["t_sel"] + res["t_prep"] + res["t_attn"]
        sums["t_dense"] += res["t_dense"]
        sums["blocks"] += res["total_blocks"]
        mq = wl.num_blocks
        sums["causal"] += wl.num_q_heads * mq * (mq + 1) // 2
    f_dense = layers * 4.0 * base.num_q_heads * base.head_dim * base.seq_len * (base.seq_len + 1) / 2
    print(json.dumps({
        "stack": wname, "layers": layers, "t_total_ms": round(sums["t_total"], 3),
        "t_estimate_ms": round(sums["t_est"], 3), "t_select_ms": round(sums["t_sel"], 3),
        "t_attention_ms": round(sums["t_attn"], 3), "t_dense_ms": round(sums["t_dense"], 3),
        "speedup_vs_dense": round(sums["t_dense"] / sums["t_total"], 3),
        "dense_equiv_tflops": round(f_dense / (sums["t_total"] * 1e-3) / 1e12, 2),
        "estimation_overhead_pct": round(100.0 * (sums["t_est"] + sums["t_sel"]) / sums["t_stages"], 2),
        "sparsity": round(1.0 - sums["blocks"] / sums["causal"], 4)}), flush=True)


def run_decoder(wname: str, layers: int, workers: int, reps: int = 1):
    """A `layers`-layer decoder prefill (DecoderPrefill) on workload `wname`'s
    shape, layer l's structured inputs drawn with seed l: the whole prefill
    timed as one region with the sparse path and again with the dense kernel,
    from the same embedding output, `reps` times each (the last is reported)."""
    import torch
    from paper_2509_24745_amd.synth import WORKLOADS
    base = WORKLOADS[wname]
    structured = []
    t = time.time()
    for layer, inputs in _layer_stream(wname, layers, workers):
        structured.append(inputs)
        print(f"[bench] decoder layer {layer}: structured inputs resident "
              f"({time.time() - t:.0f} s)", file=sys.stderr, flush=True)
    dec = DecoderPrefill(base, structured)
    x0 = dec.embed()
    for dense in (False, True):                       # warm-up: layer 0 both ways
        dec.layer(0, x0, dense)
    torch.cuda.synchronize()
    blocks = []

    def count(_):
        blocks.append(dec.bufs.block_count.sum())

    for rep in range(reps):
        blocks.clear()
        xs, (t_sp, a_sp) = dec.forward(x0, dense=False, timed=True, hook=count)
        print(f"[bench] decoder sparse prefill {t_sp:.1f} ms (attention {a_sp:.1f})",
              file=sys.stderr, flush=True)
        xd, (t_dn, a_dn) = dec.forward(x0, dense=True, timed=True)
        print(f"[bench] decoder dense prefill {t_dn:.1f} ms (attention {a_dn:.1f})",
              file=sys.stderr, flush=True)
        if rep + 1 < reps:
            del xs, xd
    mq = base.num_blocks
    causal = base.num_q_heads * mq * (mq + 1) // 2
    sp = [1.0 - int(c) / causal for c in blocks]
    diff = float((xs.float() - xd.float()).norm() / xd.float().norm())
    print(json.dumps({
        "ttft_decoder": wname, "layers": layers, "hidden": dec.hidden,
        "intermediate": dec.inter, "alpha": dec.alpha,
        "ttft_sparse_ms": round(t_sp, 1), "ttft_dense_ms": round(t_dn, 1),
        "ttft_speedup": round(t_dn / t_sp, 3),
        "attention_sparse_ms": round(a_sp, 1), "attention_dense_ms": round(a_dn, 1),
        "attention_speedup": round(a_dn / a_sp, 3),
        "nonattn_sparse_ms": round(t_sp - a_sp, 1), "nonattn_dense_ms": round(t_dn - a_dn, 1),
        "attention_share_dense": round(a_dn / t_dn, 3),
        "attention_share_sparse": round(a_sp / t_sp, 3),
        "sparsity_mean": round(float(np.mean(sp)), 4),
        "sparsity_min_max": [round(min(sp), 4), round(max(sp), 4)],
        "final_hidden_rel_diff": round(diff, 5)}), flush=True)


W128 = "llama3_8b_n131072"
SWEEPS = {
    # the 128K layer over thresholds and head similarity
    "gamma_sigma_128k": [(W128, dict(gamma=g, noise=s), "dynamic")
                         for s in (0.1, 0.3, 0.6) for g in (0.9, 0.95, 0.99)],
    # the 32K layer
    "llama_32k": [("llama3_8b_n32768", {}, "dynamic")],
    # heterogeneous Qwen-shaped layer over proxy groups and minimum budgets
    "qwen_64k": [("qwen25_7b_n65536", dict(num_proxy_groups=g, min_budget_tokens=mb), "dynamic")
                 for g in (1, 2, 4, 7) for mb in (0, 2048)],
    # one layer of the 256K 32-layer stack (layer 0)
    "llama_256k_layer": [("llama3_8b_n262144", {}, "dynamic")],
    # budget allocation at 128K: per-head dynamic budgets (constant and
    # per-row-ratio readings of Eq. 3) against a static Top-K with the same
    # mean budget, at three thresholds
    "budget_variants_128k": [(W128, dict(gamma=g), v) for g in (0.9, 0.95, 0.99)
                             for v in ("dynamic", "row_ratio", "static_match")],
    # estimation stride, minimum budget and number of proxy heads at 128K
    "stride_128k": [(W128, dict(stride=st), "dynamic") for st in (1, 2, 4)],
    "min_budget_128k": [(W128, dict(min_budget_tokens=mb), "dynamic") for mb in (0, 1024, 2048)],
    "groups_128k": [(W128, dict(num_proxy_groups=g), "dynamic") for g in (1, 2, 4, 8)],
    # the Llama-shaped layer over sequence lengths (same recipe and seed)
    "seq_len_llama": [("llama3_8b_n32768", dict(seq_len=n, name=f"llama3_8b_n{n}"), "dynamic")
                      for n in (8192, 16384, 32768, 65536, 131072, 262144)],
    # head similarity (Eq. 4 overlap of the last token, top 1024) against the
    # per-head deviation, beside the path's timing and recall
    "head_similarity_128k": [(W128, dict(noise=sg), "dynamic+overlap") for sg in (0.1, 0.3, 0.6)],
}


def run_shard(wname: str, parts: int, steps: int, warmup: int, dense_steps: int):
    """Head sharding, timed on one GPU: the layer of workload `wname` with one
    proxy group per KV head (G = Hkv), whole and in `parts` parts of Hq/P
    query heads and Hkv/P KV heads.  Each part runs the path on its own
    slices of Q, K and V, as one of P GPUs would, with no data from the
    others (the part's results are those heads' results of the whole layer;
    tests/test_gpu_shard.py checks that).  Prints one JSON line: the whole
    step, every part's step, and the parallel efficiency the slowest part
    allows, (whole / P) / slowest part."""
    from paper_2509_24745_amd.synth import WORKLOADS
    base = WORKLOADS[wname]
    if parts < 1 or base.num_kv_heads % parts:
        raise SystemExit(f"--shard: the parts must divide the {base.num_kv_heads} KV heads")
    wl = base.replace(num_proxy_groups=base.num_kv_heads)
    full, _, (q, k, v) = measure(wl, steps, warmup, dense_steps, with_dense=True)
    rq, rk, rg = wl.num_q_heads // parts, wl.num_kv_heads // parts, wl.num_proxy_groups // parts
    res = []
    for s in range(parts):
        sl = (q[:, s * rq:(s + 1) * rq].contiguous(), k[:, s * rk:(s + 1) * rk].contiguous(),
              v[:, s * rk:(s + 1) * rk].contiguous())
        ws = wl.replace(num_q_heads=rq, num_kv_heads=rk, num_proxy_groups=rg,
                        name=f"{wl.name}_part{s}of{parts}")
        r, _, _ = measure(ws, steps, warmup, dense_steps, with_dense=False, inputs=sl)
        res.append(r)
        del sl
    t_parts = [r["ms_total"] for r in res]
    print(json.dumps({
        "shard": wl.name, "parts": parts, "num_proxy_groups": wl.num_proxy_groups,
        "part_heads": [rq, rk, rg], "t_whole_ms": round(full["ms_total"], 3),
        "t_part_ms": [round(t, 3) for t in t_parts], "t_part_max_ms": round(max(t_parts), 3),
        "t_whole_over_parts_ms": round(full["ms_total"] / parts, 3),
        "parallel_efficiency": round(full["ms_total"] / parts / max(t_parts), 3),
        "t_dense_whole_ms": round(full["t_dense"], 3),
        "speedup_vs_dense_sharded": round(full["t_dense"] / parts / max(t_parts), 3),
        "sparsity_whole": round(full["sparsity"], 4),
        "sparsity_parts": [round(r["sparsity"], 4) for r in res],
        "attn_mfma_frac_parts": [round(r["achieved"] / r["peak"], 4) for r in res]}), flush=True)


def overlap_stats(wl, inputs, topk: int = 1024):
    """Eq. 4 overlap matrices of the last query token on the GPU, summarised:
    mean over pairs of different heads, split into pairs sharing a KV head
    and pairs that do not; raw, sinks (4 tokens) removed, and renormalised."""
    import torch
    from paper_2509_24745_amd import proxyattn as pa
    prob = pa.Problem(seq_len=wl.seq_len, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                      head_dim=wl.head_dim, block_size=wl.block_size,
                      num_proxy_groups=wl.num_proxy_groups, stride=wl.stride, dtype=wl.dtype)
    q, k, _ = inputs
    ws = torch.empty(pa.proxyattn_workspace_size(prob), dtype=torch.uint8, device="cuda")
    hq, rep = wl.num_q_heads, wl.num_q_heads // wl.num_kv_heads
    scores = torch.empty((hq, hq), dtype=torch.float32, device="cuda")
    grp = np.arange(hq) // rep
    same = (grp[:, None] == grp[None, :]) & ~np.eye(hq, dtype=bool)
    cross = grp[:, None] != grp[None, :]
    out = {}
    for tag, sink, renorm in (("raw", 0, False), ("no_sink", 4, False), ("no_sink_renorm", 4, True)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        pa.proxyattn_head_overlap(prob, q, k, wl.seq_len - 1, topk, sink, renorm, scores, ws)
        e1.record()
        torch.cuda.synchronize()
        sc = scores.cpu().numpy().astype(np.float64)
        out[tag] = {"same_kv_mean": round(float(sc[same].mean()), 4),
                    "cross_kv_mean": round(float(sc[cross].mean()), 4),
                    "self_mean": round(float(np.diag(sc).mean()), 4), "ms": round(e0.elapsed_time(e1), 3)}
    return out


def input_key(wname: str, wl) -> tuple:
    """Identity of a workload's generated inputs: every field that changes the
    tensors (their shape and the generator settings), none that only changes
    the method's arguments (gamma, G, stride, budgets).  Sweep points with equal
    keys share one upload."""
    return (wname, wl.seq_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.dtype,
            wl.structure, wl.seed)


def run_sweep(name: str, steps: int, warmup: int, dense_steps: int):
    from paper_2509_24745_amd.synth import WORKLOADS
    cache = {}       # device inputs of the current generator settings
    dense = {}       # dense time and lse per generator settings
    last_mean = {}   # mean dynamic budget per (workload, settings) for static_match
    for wname, kw, variant in SWEEPS[name]:
        wl = WORKLOADS[wname].replace(**kw) if kw else WORKLOADS[wname]
        key = input_key(wname, wl)
        static_k = None
        with_overlap = variant.endswith("+overlap")
        variant = variant.replace("+overlap", "")
        if variant == "static_match":
            variant = "static"
            static_k = max(1, int(round(last_mean[(key, wl.gamma, wl.min_budget_tokens)])))
        d = dense.get(key)
        # shorter sequences take more steps, so that every point's timed
        # region is about as long as the 128K point's (host launch latency
        # and clock ramp-up otherwise show in a region of a few milliseconds)
        n_steps = min(1000, max(steps, int(steps * (131072 / wl.seq_len) ** 2)))
        n_dense = min(200, max(dense_steps, int(dense_steps * (131072 / wl.seq_len) ** 2)))
        res, host, inputs = measure(wl, n_steps, warmup, n_dense, with_dense=d is None,
                                    inputs=cache.get(key), variant=variant, static_k=static_k,
                                    dense_lse=d["lse"] if d else None)
        cache = {key: inputs}
        if d is None:
            dense = {key: {"t": res["t_dense"], "frac": res["dense_mfma_frac"],
                           "lse": res["dense_lse"]}}
        else:
            res["t_dense"], res["dense_mfma_frac"] = d["t"], d["frac"]
        if variant == "dynamic":
            last_mean[(key, wl.gamma, wl.min_budget_tokens)] = res["head_count_mean"]
        line = summary_line(wl, res, n_steps)
        if with_overlap:
            line["head_overlap_top1024"] = overlap_stats(wl, inputs)
        print(json.dumps(line), flush=True)


# The paper's own speedups (Sec. 4.3, Efficiency Results, with Fig. 4 for the
# attention kernel and Fig. 1 for prefill), printed beside the measured ones
# for context: other hardware, and real model activations from RULER, which
# the synthetic inputs here only stand in for.
PAPER_CONTEXT = {
    "attention_speedup_vs_flashattention": 10.3, "attention_tokens": 262144,
    "prefill_ttft_speedup": 2.4, "prefill_tokens": 131072,
    "hardware": "NVIDIA H800-80GB", "inputs": "RULER activations of real models",
    "note": "context only: not the same hardware, inputs or baseline kernel",
}


# (attn_order, attn_chunk_rows) points of --work-orders (problem descriptor
# fields): 1 = longest rows first, heads fastest; 2 = chunks of R rows x all
# heads; 3 = chunks of R rows x the query heads of one KV head, KV head by KV
# head.
WORK_ORDERS = [(1, 1), (2, 2), (2, 8), (3, 1), (3, 4), (3, 16), (3, 64)]


def run_work_orders(wl, reps: int):
    """Time the block-sparse call on one set of lists under each work-item
    order of the library (the problem's attn_order / attn_chunk_rows), one
    JSON line per order.  Launch sequence, which a rocprofv3
    --pmc run of this mode sees in the same order: per order one untimed call,
    then `reps` timed calls."""
    import torch
    from paper_2509_24745_amd import proxyattn as pa
    from paper_2509_24745_amd.synth import generate

    prob = pa.Problem(seq_len=wl.seq_len, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                      head_dim=wl.head_dim, block_size=wl.block_size,
                      num_proxy_groups=wl.num_proxy_groups, stride=wl.stride, dtype=wl.dtype)
    host = generate(wl)
    q, k, v = (torch.from_numpy(host[x]).to(prob.torch_dtype).cuda() for x in ("q", "k", "v"))
    del host
    bufs = pa.Buffers(prob)
    st = torch.cuda.current_stream()
    pa.proxyattn_estimate(prob, q, k, bufs.logscore, bufs.mass, bufs.workspace, st)
    pa.proxyattn_select_budget(prob, bufs.logscore, bufs.mass, wl.gamma, wl.min_budget_tokens,
                               bufs.head_count, bufs.block_count, bufs.block_index, st)
    torch.cuda.synchronize()
    blocks = int(bufs.block_count.sum().item())
    for order, rows in WORK_ORDERS:
        po = dataclasses.replace(prob, attn_order=order, attn_chunk_rows=rows)
        call = lambda: pa.proxyattn_block_sparse_prefill(
            po, q, k, v, bufs.block_count, bufs.block_index, bufs.out, None, bufs.workspace, st)
        call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            call()
        e1.record(st)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        print(json.dumps({"workload": wl.name, "attn_order": order, "chunk_rows": rows,
                          "attn_ms": round(ms, 3), "reps": reps, "computed_blocks": blocks,
                          "attn_tflops": round(4.0 * wl.block_size ** 2 * wl.head_dim *
                                               blocks / (ms * 1e-3) / 1e12, 1)}),
              flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU: --gpus must be 1 (the path "
                                   "shards by heads across GPUs only by design)"}))
        sys.exit(2)
    if args.profile_summary:
        print(profile_summary(args.profile_summary, args.workload), end="")
        return
    import torch
    if args.calibrate_copy:
        n = 1 << 30
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        a.fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n}))
        return
    from paper_2509_24745_amd.synth import WORKLOADS
    if args.shard:
        run_shard(args.workload, args.shard, args.steps, args.warmup, args.dense_steps)
        return
    if args.stack and args.ttft:
        run_decoder(args.workload, args.stack, args.stack_workers)
        return
    if args.stack:
        run_stack(args.workload, args.stack, args.steps, args.warmup, args.dense_steps,
                  args.stack_workers)
        return
    if args.sweep:
        run_sweep(args.sweep, args.steps, args.warmup, args.dense_steps)
        return
    if args.work_orders:
        run_work_orders(WORKLOADS[args.workload], max(1, args.steps))
        return

    wl = WORKLOADS[args.workload]
    kw = {}
    if args.gamma is not None:
        kw["gamma"] = args.gamma
    if args.noise is not None:
        kw["noise"] = args.noise
    if args.num_proxy_groups is not None:
        kw["num_proxy_groups"] = args.num_proxy_groups
    if args.min_budget is not None:
        kw["min_budget_tokens"] = args.min_budget
    if args.seq_len is not None:
        kw["seq_len"] = args.seq_len
        kw["name"] = f"{wl.name.rsplit('_n', 1)[0]}_n{args.seq_len}"
    wl = wl.replace(**kw) if kw else wl
    r, g, dev_inputs = measure(wl, args.steps, args.warmup, args.dense_steps,
                               with_dense=not args.no_dense)
    t_vendor = None if args.no_dense or wl.dtype != "bf16" else vendor_dense_ms(wl, dev_inputs)
    del dev_inputs
    ms_total, t_est, t_sel, t_attn, t_dense = r["ms_total"], r["t_est"], r["t_sel"], r["t_attn"], r["t_dense"]
    n, hq, d, b = wl.seq_len, wl.num_q_heads, wl.head_dim, wl.block_size
    mq = wl.num_blocks
    sparsity, total_blocks, f_dense, achieved, peak = (r["sparsity"], r["total_blocks"], r["f_dense"],
                                                       r["achieved"], r["peak"])

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, g["q"], g["k"], g["v"], args.cpu_sample_rows)

    line = {
        "metric": METRIC,
        "value": round(ms_total, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_total, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "seq_len": n, "num_q_heads": hq,
                   "num_kv_heads": wl.num_kv_heads, "head_dim": d, "block_size": b,
                   "num_proxy_groups": wl.num_proxy_groups, "stride": wl.stride,
                   "gamma": wl.gamma, "head_deviation": wl.structure.noise,
                   "min_budget_tokens": wl.min_budget_tokens, "parallelism": "single GPU"},
        "t_estimate_ms": round(t_est, 4),
        "t_select_ms": round(t_sel, 4),
        "t_prepare_kv_ms": round(r["t_prep"], 4),
        "t_attention_ms": round(t_attn, 4),
        "step_ms_median": round(r["step_median"], 4) if r["step_median"] is not None else None,
        "step_ms_min": round(r["step_min"], 4) if r["step_min"] is not None else None,
        "graph_replay_ms_per_step": round(r["t_graph"], 4) if r["t_graph"] else None,
        "torch_sdpa_flash_ms": round(t_vendor, 3) if t_vendor else None,
        "speedup_vs_torch_sdpa_flash": round(t_vendor / ms_total, 3) if t_vendor else None,
        "dense_equiv_tflops": round(f_dense / (ms_total * 1e-3) / 1e12, 2),
        "estimation_overhead_pct": round(100.0 * r["est_share"], 2),
        "sparsity": round(sparsity, 4),
        "t_dense_ms": round(t_dense, 4) if t_dense else None,
        "t_dense_attention_ms": round(r["t_dense_attn"], 4) if t_dense else None,
        "speedup_vs_dense": round(t_dense / ms_total, 3) if t_dense else None,
        "estimation_overhead_pct_of_dense": round(100.0 * (t_est + t_sel) / t_dense, 2)
        if t_dense else None,
        "dense_mfma_frac": round(r["dense_mfma_frac"], 4) if t_dense else None,
        "computed_blocks": total_blocks,
        "attention_mass_recall": ({k: round(x, 5) for k, x in r["recall"].items()}
                                  if r["recall"] else None),
        "roofline": {"kernel": "attn_kernel (block-sparse blocked prefill call)", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic() if wl.name == "llama3_8b_n131072" and
                     wl.gamma == 0.95 and wl.structure.noise == 0.3 else None},
        "cpu_baseline": cpu,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
