#!/usr/bin/env python3
"""Benchmark of draft-step attention over reused target KV on one MI355X.

Default workload: batch 64, target context 32768, 32 query / 8 KV heads,
head_dim 128, k = 8 draft steps folded into one call, bf16, 16-token pages
with a random page table.  One "step" is one pass of the whole path over that
batch: the attention kernel plus, when the context is split, the combine
kernel (``--mode sequential`` makes a step k calls of one draft query each).

Prints one JSON line: effective HBM GB/s (algorithmic bytes / step time),
draft tokens/s, the roofline of the dominant (attention) kernel, and the CPU
oracle timed on a bounded sample of the same workload.  Other workloads
(``--workload``) print the same fields.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads.device as WD  # noqa: E402  (seeded inputs only)

PEAK_HBM_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
METRIC = "draft-attention effective HBM GB/s (% of peak) + draft tokens/s at 32K ctx"
DEFAULT_WORKLOAD = "long_b64_ctx32k_k8"
# bf16 parity bars against the float64 oracle (the parity sample must meet both)
PARITY_MAX_ABS = 2e-2
PARITY_REL_L2 = 5e-3


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


KERNEL_SOURCES = {1: ("attn_mfma.hip", "attn_mfma_common.h", "kvshot_common.h"),
                  3: ("attn_tall.hip", "attn_mfma_common.h", "kvshot_common.h")}
KERNEL_NAMES = {1: "attn_mfma_kernel", 2: "attn_generic_kernel", 3: "attn_tall_kernel"}
PROFILE_PREFIX = {1: "attn_mfma", 3: "attn_tall"}


def kernel_source_hash(path: int = 1) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[path]:
        h.update(open(os.path.join(ROOT, "paper_2604_26412_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(workload: str, mode: str, kernel_path: int = 1):
    """HBM bytes per attention launch from a committed counter summary, if it matches this kernel source."""
    if kernel_path not in PROFILE_PREFIX:
        return None
    path = os.path.join(PROFILES, f"{PROFILE_PREFIX[kernel_path]}_{workload}_{mode}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    f = re.search(r"fetch_bytes_per_launch:\s*([0-9.eE+]+)", text)
    w = re.search(r"write_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m and f and w) or m.group(1) != kernel_source_hash(kernel_path):
        return None
    return float(f.group(1)) + float(w.group(1))


# ---------------------------------------------------------------------------
# workloads on the device
# ---------------------------------------------------------------------------

def upload_case(torch, case):
    import numpy as np

    def dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()
    B, n, Hq, D = case.q.shape
    extra = case.step_offsets if case.mode == "step" else case.parents
    return dict(mode=case.mode, q=dev(case.q), k_pages=dev(case.k_pages), v_pages=dev(case.v_pages),
                page_table=dev(case.page_table), ctx_lens=dev(case.ctx_lens), draft_k=dev(case.draft_k),
                draft_v=dev(case.draft_v), extra=dev(extra), pool=case.num_pages, pps=case.max_pages_per_seq, B=B,
                n=n, Hq=Hq, Hkv=case.num_kv_heads, D=D, P=case.page_size, max_draft=case.max_draft,
                lens=[int(x) for x in case.ctx_lens], dtype=case.dtype, host=case, theta=case.rope_theta,
                scale=case.softmax_scale,
                offsets=[int(x) for x in case.step_offsets] if case.mode == "step" else [0] * B)


# ---------------------------------------------------------------------------
# byte accounting
# ---------------------------------------------------------------------------

def call_bytes(d, n_q, draft_seen):
    """Algorithmic bytes of one call: target K/V once, page-table entries, q, draft K/V seen, out."""
    eb = 2 if d["dtype"] == "bf16" else 4
    row = d["Hkv"] * d["D"] * eb
    kv = sum(2 * T * row for T in d["lens"])
    pt = sum(-(-T // d["P"]) * 4 for T in d["lens"])
    q = d["B"] * n_q * d["Hq"] * d["D"] * eb
    dkv = sum(2 * s * row for s in draft_seen)
    return kv + pt + q + dkv + q


def copy_calibration(torch, gib: float):
    """One plain device copy of `gib` GiB: the reference a profiler's byte counters are scaled by."""
    if gib <= 0:
        return
    nbytes = int(gib * (1 << 30))
    src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: {nbytes} bytes read and written by one copy kernel")
    del src, dst


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return int(os.environ.get("OMP_NUM_THREADS", "1"))


def cpu_baseline(torch, d, out_gpu, budget_s=20.0):
    """Time the float64 oracle on a bounded sample of whole sequences of the same workload: as many as
    fit the budget at the first sequence's rate, up to the whole batch."""
    import numpy as np

    import oracle

    def sample(seqs):
        if d["host"] is None:
            return WD.host_sample(torch, d, seqs), None
        return d["host"], seqs

    c0, s0 = sample([0])
    t0 = time.perf_counter()
    ref0, _ = oracle.draft_attention(c0, seqs=s0)
    t1 = time.perf_counter() - t0
    if s0 is not None:
        ref0 = ref0[[0]]
    ns = int(max(0, min(d["B"] - 1, budget_s // max(t1, 1e-3))))
    if ns == 0:                                    # one sequence: the first timing is the sample
        seqs, ref, dt, ns_t, timed = [], ref0[:0], t1, 1, [0]
    else:
        seqs = list(range(1, 1 + ns))
        c1, s1 = sample(seqs)
        t0 = time.perf_counter()
        ref, _ = oracle.draft_attention(c1, seqs=s1)
        dt = time.perf_counter() - t0
        if s1 is not None:
            ref = ref[seqs]
        ns_t, timed = ns, seqs
    ns = ns_t
    sub = dict(d, B=ns, lens=[d["lens"][s] for s in timed])
    if d["mode"] == "step":
        seen = [d["offsets"][s] + d["n"] for s in timed]
    else:
        seen = [d["n"]] * ns
    nbytes = call_bytes(sub, d["n"], seen)
    got = out_gpu[[0] + seqs].float().cpu().numpy().astype(np.float64)
    allref = np.concatenate([ref0, ref], 0)
    diff = got - allref
    parity = dict(max_abs=float(np.abs(diff).max()),
                  rel_l2=float(np.linalg.norm(diff) / np.linalg.norm(allref)), sequences=1 + ns)
    return dict(value=round(nbytes / dt / 1e9, 4), unit="GB/s", draft_tokens_per_s=round(ns * d["n"] / dt, 2),
                cores=blas_threads(), kind="oracle", host_cpus=os.cpu_count(), seconds=round(dt, 3),
                sample=f"{ns} whole sequence(s) of the same workload ({d['n']} draft queries x {d['Hq']} heads each)"
                       f"{' (with the first, timed apart: the whole batch)' if ns + 1 == d['B'] else ''}, "
                       f"float64 NumPy oracle; value is the same algorithmic bytes per second"), parity


def stream_ceiling(torch, K, tensor):
    """Non-temporal streaming-read rate of the device over `tensor` (GB/s)."""
    sink = torch.empty(4096 * 4, dtype=torch.int32, device="cuda")
    for _ in range(3):
        K.stream_read(tensor, sink, 4096)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        K.stream_read(tensor, sink, 4096)
    e1.record()
    torch.cuda.synchronize()
    return tensor.numel() * tensor.element_size() / (e0.elapsed_time(e1) / 10 * 1e-3) / 1e9


def mfma_ceiling(torch, K, iters: int = 4096):
    """Dense bf16 matrix rate the whole chip sustains (TFLOP/s): ten back-to-back launches of the
    library's matrix-rate probe, about 1 ms each, one workgroup of four waves per CU."""
    wgs = torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.empty(wgs * 4, dtype=torch.int32, device="cuda")
    for _ in range(3):
        K.mfma_rate(iters, wgs, sink)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        K.mfma_rate(iters, wgs, sink)
    e1.record()
    torch.cuda.synchronize()
    flops = wgs * 4 * iters * 16 * 32768.0
    return flops / (e0.elapsed_time(e1) / 10 * 1e-3) / 1e12


def add_mfma_ceiling(torch, K, roof):
    """For a matrix-bound kernel, the measured sustained matrix rate beside the published peak."""
    if roof["bound"] != "mfma":
        return
    ceil = mfma_ceiling(torch, K)
    roof["measured_mfma_ceiling"] = round(ceil, 1)
    roof["frac_of_measured_ceiling"] = round(roof["achieved"] / ceil, 4)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--op", choices=["attention", "fusion", "kvproj", "accept", "treegrow"], default="attention",
                    help="attention: the draft-step attention path (default); fusion: the hybrid drafter's "
                         "gated delta fusion; kvproj: the projected-KV cache builder of KV-only drafters; "
                         "accept: acceptance rates and MAT over verification records; treegrow: level-wise "
                         "draft-tree growth from the drafter's logits")
    ap.add_argument("--workload", default=None,
                    choices=[DEFAULT_WORKLOAD, "tree_b8_ctx16k_n60", "ragged_b16_k6", "single_ctx4096_k8",
                             "fusion_t64_d4096", "fusion_t480_d4096", "kvproj_prefill_b64_t32k",
                             "kvproj_verify_b64_t32k", "accept_n64m_k7", "treegrow_b8_v152k_d8k10n60"])
    ap.add_argument("--no-rope", action="store_true", help="--op kvproj: plain projection (no RoPE on keys)")
    ap.add_argument("--fusion-tile", type=int, default=0, choices=[0, 1, 2],
                    help="--op fusion: token tile, 0 automatic, 1 64 tokens, 2 128 tokens")
    ap.add_argument("--kvproj-path", type=int, default=0, choices=[0, 1, 2],
                    help="--op kvproj: 0 automatic, 1 the tiled kernel, 2 the direct kernel")
    ap.add_argument("--mode", choices=["folded", "sequential"], default="folded")
    ap.add_argument("--splits", type=int, default=0)
    ap.add_argument("--contiguous", action="store_true",
                    help="64 x 32K workload: contiguous page table instead of a random permutation")
    ap.add_argument("--calls", type=int, default=None,
                    help="per-call timing sample for the median and p10/p90 (default: 100 for the 64 x 32K "
                         "workload, 200 otherwise; 0 skips it)")
    ap.add_argument("--path", choices=["auto", "mfma", "generic", "general-mfma"], default="auto",
                    help="attention kernel: the planner's choice (bf16: MFMA, 256-row tiles on the tall-tile "
                         "kernel), or forced; general-mfma: the general MFMA kernel for every tile height")
    ap.add_argument("--cold", action="store_true",
                    help="flush the device caches (write 1 GiB) before every timed call; per-call events")
    ap.add_argument("--no-graph", action="store_true",
                    help="launch each step from Python instead of replaying a captured HIP graph of it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=1004)
    ap.add_argument("--fusion-row-major", action="store_true",
                    help="--op fusion: read the weights in their row-major layout instead of the packed copy")
    ap.add_argument("--copy-calib-gib", type=float, default=0.0,
                    help="also run one plain device copy of this many GiB (counter calibration under a profiler)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2604_26412_amd as K
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.op == "fusion":
        return bench_fusion(args, torch, K, W)
    if args.op == "kvproj":
        return bench_kvproj(args, torch, K, W)
    if args.op == "accept":
        return bench_accept(args, torch, K, W)
    if args.op == "treegrow":
        return bench_treegrow(args, torch, K, W)
    if args.workload is None:
        args.workload = DEFAULT_WORKLOAD
    if args.workload.startswith("fusion"):
        raise SystemExit("fusion workloads run with --op fusion")
    if args.workload == DEFAULT_WORKLOAD:
        log("generating the 64 x 32768 workload on the device")
        d = WD.long_range_on_device(torch, args.seed, contiguous=args.contiguous)
    elif args.contiguous:
        raise SystemExit("--contiguous applies to the 64 x 32K workload only")
    else:
        log(f"generating {args.workload} on the host")
        d = upload_case(torch, W.workload(args.workload))
    if d["mode"] == "tree" and args.mode == "sequential":
        raise SystemExit("sequential mode applies to step workloads only")
    torch.cuda.synchronize()
    B, n, Hq, Hkv, D, P = d["B"], d["n"], d["Hq"], d["Hkv"], d["D"], d["P"]
    T_max = max(d["lens"])
    att = K.DraftAttention(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, page_size=P, dtype=d["dtype"],
                           max_batch=B, max_draft=d["max_draft"], max_pages_per_seq=d["pps"], num_pages=d["pool"],
                           rope_theta=d["theta"], softmax_scale=d["scale"])
    if args.splits:
        att.set_option(K.OPT_SPLITS, args.splits)
    if args.path != "auto":
        att.set_option(K.OPT_PATH, {"mfma": 1, "generic": 2, "general-mfma": 3}[args.path])
    nq_call = n if args.mode == "folded" else 1
    plan = att.plan(B, nq_call, T_max)
    edt = torch.bfloat16 if d["dtype"] == "bf16" else torch.float32
    out = torch.empty((B, n, Hq, D), dtype=edt, device="cuda")
    stream = torch.cuda.current_stream()

    if d["mode"] == "tree":
        def step():
            att.tree(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["ctx_lens"], d["draft_k"], d["draft_v"],
                     d["extra"], max_ctx=T_max, out=out)
        draft_seen = [[n] * B]
    elif args.mode == "folded":
        def step():
            att.step(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["ctx_lens"], d["draft_k"], d["draft_v"],
                     d["extra"], max_ctx=T_max, out=out)
        draft_seen = [[o + n for o in d["offsets"]]]
    else:
        qs = [d["q"][:, j:j + 1].contiguous() for j in range(n)]
        offs = [(d["extra"] + j).contiguous() for j in range(n)]
        outs = [torch.empty((B, 1, Hq, D), dtype=edt, device="cuda") for _ in range(n)]

        def step():
            for j in range(n):
                att.step(qs[j], d["k_pages"], d["v_pages"], d["page_table"], d["ctx_lens"], d["draft_k"],
                         d["draft_v"], offs[j], max_ctx=T_max, out=outs[j])
        draft_seen = [[o + j + 1 for o in d["offsets"]] for j in range(n)]
    step_bytes = sum(call_bytes(d, nq_call, seen) for seen in draft_seen)
    # the attention kernel of the last call of a step; with split-K the combine writes the output
    out_bytes = B * nq_call * Hq * D * (2 if d["dtype"] == "bf16" else 4)
    attn_launch_bytes = call_bytes(d, nq_call, draft_seen[-1]) - (out_bytes if plan["splits"] > 1 else 0)

    copy_calibration(torch, args.copy_calib_gib)

    log(f"plan {plan}; warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run_step = step
    if not args.no_graph:
        # capture one step (every kernel launch of the path) in a HIP graph and replay it
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run_step = graph.replay
        for _ in range(args.warmup):
            run_step()
        torch.cuda.synchronize()
    log(f"timing {args.steps} steps" + (" (cold caches)" if args.cold else ""))
    if args.cold:
        flush = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
        times = []
        for _ in range(args.steps):
            flush.fill_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            run_step()
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        times.sort()
        ms_per_step = times[len(times) // 2]
        del flush
    else:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            run_step()
        e1.record(stream)
        torch.cuda.synchronize()
        ms_per_step = e0.elapsed_time(e1) / args.steps

    # per-call distribution: each replay between its own pair of events (median, p10, p90)
    ncalls = args.calls if args.calls is not None else (100 if args.workload == DEFAULT_WORKLOAD else 200)
    call_ms = None
    if ncalls > 0 and not args.cold:
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(ncalls)]
        torch.cuda.synchronize()
        for a, z in evs:
            a.record(stream)
            run_step()
            z.record(stream)
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(z) for a, z in evs)
        call_ms = {"calls": ncalls, "median": round(ts[ncalls // 2], 5), "p10": round(ts[ncalls // 10], 5),
                   "p90": round(ts[(9 * ncalls) // 10], 5)}
        log(f"per call over {ncalls}: median {call_ms['median']:.4f} ms, p10 {call_ms['p10']:.4f}, "
            f"p90 {call_ms['p90']:.4f}")

    # per-kernel durations from HIP events the library records around each launch on this stream
    att.set_option(K.OPT_PROFILE, 1)
    for _ in range(args.steps):
        step()
    prof = att.profile_read()
    att.set_option(K.OPT_PROFILE, 0)
    calls = max(1, prof["calls"])
    attn_ms = prof["attn_ms"] / calls
    comb_ms = prof["combine_ms"] / calls
    log(f"step {ms_per_step:.4f} ms; attention kernel {attn_ms:.4f} ms; combine {comb_ms:.4f} ms")
    ceiling = stream_ceiling(torch, K, d["k_pages"])
    log(f"non-temporal streaming-read ceiling {ceiling:.1f} GB/s")

    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    achieved = attn_launch_bytes / (attn_ms * 1e-3) / 1e9
    traffic = read_traffic(args.workload, args.mode, plan["path"]) if not args.splits else None
    path_name = KERNEL_NAMES[plan["path"]]
    kernel = f"{path_name} ({plan['row_tiles']} x 32-row query tiles per (sequence, KV head))" \
        if plan["path"] != 2 else path_name
    res = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "pct_of_peak": round(100.0 * value / PEAK_HBM_GBS, 2),
        "draft_tokens_per_s": round(B * n / (ms_per_step * 1e-3), 1),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": d["dtype"],
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: batch {B}, ctx {T_max if len(set(d['lens'])) == 1 else 'ragged'}, "
                               f"{Hq}/{Hkv} heads, head_dim {D}, {n} draft "
                               f"{'nodes (tree)' if d['mode'] == 'tree' else 'steps (' + args.mode + ')'}, "
                               f"{d['dtype']}, {P}-token pages, random page table",
                   "batch": B, "ctx_len_max": T_max, "draft_queries": n, "mode": args.mode if d["mode"] == "step"
                   else "tree", "page_size": P, "splits": plan["splits"], "workgroups": plan["workgroups"],
                   "cold_caches": bool(args.cold), "launch": "python" if args.no_graph else "hip graph replay",
                   "path": {1: "mfma", 2: "generic", 3: "mfma (tall tiles)"}[plan["path"]],
                   "page_table": "contiguous" if args.contiguous else "random permutation"},
        "call_ms": call_ms,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic, "kernel": kernel,
                     "kernel_ms": round(attn_ms, 5), "combine_ms": round(comb_ms, 5),
                     "algorithmic_bytes_per_launch": attn_launch_bytes,
                     "measured_stream_read_ceiling": round(ceiling, 1),
                     "frac_of_measured_ceiling": round(achieved / ceiling, 4)},
        "whole_job_algorithmic_bytes": step_bytes,
    }
    if not args.no_cpu_baseline and args.mode == "folded":
        log("timing the CPU oracle on a bounded sample")
        cb, parity = cpu_baseline(torch, d, out)
        res["cpu_baseline"] = cb
        parity["ok"] = parity["max_abs"] <= PARITY_MAX_ABS and parity["rel_l2"] <= PARITY_REL_L2
        res["parity_sample"] = parity
    print(json.dumps(res), flush=True)
    att.close()
    if "parity_sample" in res and not res["parity_sample"]["ok"]:
        log(f"parity sample misses the bars (max-abs <= {PARITY_MAX_ABS}, rel-L2 <= {PARITY_REL_L2}): "
            f"{res['parity_sample']}")
        sys.exit(1)


# ---------------------------------------------------------------------------
# gated delta fusion (--op fusion)
# ---------------------------------------------------------------------------

PEAK_BF16_TFLOPS = 2500.0
FUSION_METRIC = "gated-delta fusion tokens/s (d=4096, bf16) with achieved TFLOP/s and HBM GB/s"


def fusion_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("fusion.hip", "fusion_common.h", "kvshot_common.h", "fusion_api.cpp"):
        h.update(open(os.path.join(ROOT, "paper_2604_26412_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_fusion_traffic(workload: str):
    path = os.path.join(PROFILES, f"fusion_kernel_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    f = re.search(r"fetch_bytes_per_launch:\s*([0-9.eE+]+)", text)
    w = re.search(r"write_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m and f and w) or m.group(1) != fusion_source_hash():
        return None
    return float(f.group(1)) + float(w.group(1))


def fusion_cpu_baseline(case, h_gpu, budget_s=10.0):
    """Time the float64 fusion oracle on a bounded sample of the workload's tokens."""
    import numpy as np

    import oracle
    import workloads as W

    dec = lambda b: W.bf16_bits_to_f32(b).astype(np.float64)
    wg, wd, bg = dec(case.w_g), dec(case.w_delta), case.b_g.astype(np.float64)
    t0 = time.perf_counter()
    ref = oracle.gated_delta_fusion(dec(case.n[:1]), dec(case.o[:1]), wg, bg, wd)
    t1 = time.perf_counter() - t0
    ns = int(max(1, min(case.tokens - 1, 64, budget_s // max(t1, 1e-3))))
    rows = list(range(1, 1 + ns))
    t0 = time.perf_counter()
    ref2 = oracle.gated_delta_fusion(dec(case.n[rows]), dec(case.o[rows]), wg, bg, wd)
    dt = time.perf_counter() - t0
    allref = np.concatenate([ref, ref2], 0)
    got = h_gpu[[0] + rows].float().cpu().numpy().astype(np.float64)
    diff = got - allref
    parity = dict(max_abs=float(np.abs(diff).max()), rel_l2=float(np.linalg.norm(diff) / np.linalg.norm(allref)),
                  tokens=1 + ns)
    return dict(value=round(ns / dt, 3), unit="tokens/s", cores=blas_threads(), kind="oracle",
                host_cpus=os.cpu_count(), seconds=round(dt, 3),
                sample=f"{ns} tokens of the same workload (weights decoded once, outside the timing), float64 "
                       f"NumPy oracle"), parity


def bench_fusion(args, torch, K, W):
    name = args.workload or "fusion_t64_d4096"
    if name not in W.FUSION_WORKLOADS:
        raise SystemExit(f"--op fusion takes one of {sorted(W.FUSION_WORKLOADS)}")
    spec = W.FUSION_WORKLOADS[name]
    log(f"generating {name} on the host")
    case = W.fusion_case(spec["tokens"], spec["d"], seed=spec["seed"])
    tokens, d = case.tokens, case.d

    def dev(a):
        import numpy as np
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()
    n, o, w_g, b_g, w_delta = dev(case.n), dev(case.o), dev(case.w_g), dev(case.b_g), dev(case.w_delta)
    h = torch.empty((tokens, d), dtype=torch.bfloat16, device="cuda")
    fz = K.GatedDeltaFusion(d, tokens)
    if args.splits:
        fz.set_option(K.OPT_SPLITS, args.splits)
    if args.fusion_tile:
        fz.set_option(K.OPT_PATH, args.fusion_tile)
    plan = fz.plan(tokens)
    # weights are packed once, as a serving engine does at load time (outside the timed region)
    packed = None if args.fusion_row_major else fz.pack_weights(w_g, w_delta)
    torch.cuda.synchronize()

    def step():
        if packed is None:
            fz(n, o, w_g, b_g, w_delta, out=h)
        else:
            fz(n, o, None, b_g, None, out=h, packed=packed)

    copy_calibration(torch, args.copy_calib_gib)

    log(f"plan {plan}; warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run_step = step
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run_step = graph.replay
        for _ in range(args.warmup):
            run_step()
        torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        run_step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps
    fz.set_option(K.OPT_PROFILE, 1)
    for _ in range(args.steps):
        step()
    prof = fz.profile_read()
    fz.set_option(K.OPT_PROFILE, 0)
    calls = max(1, prof["calls"])
    main_ms, comb_ms = prof["main_ms"] / calls, prof["combine_ms"] / calls
    log(f"step {ms_per_step:.4f} ms; fusion kernel {main_ms:.4f} ms; combine {comb_ms:.4f} ms")

    alg = W.fusion_algorithmic(tokens, d)
    out_bytes = tokens * d * 2
    part_bytes = plan["splits"] * tokens * d * 8 if plan["splits"] > 1 else 0
    # main kernel: weights, bias and activations in; the output (one split) or the split partials out
    main_bytes = alg["bytes"] - out_bytes + (part_bytes if part_bytes else out_bytes)
    intensity = alg["flops"] / alg["bytes"]
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    if intensity >= ridge:
        roof = {"bound": "mfma", "achieved": round(alg["flops"] / (main_ms * 1e-3) / 1e12, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(main_bytes / (main_ms * 1e-3) / 1e9, 2), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    add_mfma_ceiling(torch, K, roof)
    roof["traffic"] = read_fusion_traffic(name) if not (args.splits or args.fusion_tile) else None
    roof.update({"kernel": f"fusion_kernel ({plan['splits']} reduction split(s), {plan['workgroups']} workgroups)",
                 "kernel_ms": round(main_ms, 5), "combine_ms": round(comb_ms, 5),
                 "algorithmic_bytes_per_launch": main_bytes, "flops_per_launch": alg["flops"],
                 "arithmetic_intensity_flop_per_byte": round(intensity, 1),
                 "achieved_tflops": round(alg["flops"] / (main_ms * 1e-3) / 1e12, 2),
                 "achieved_gbs": round(main_bytes / (main_ms * 1e-3) / 1e9, 2)})
    res = {
        "metric": FUSION_METRIC,
        "value": round(tokens / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{name}: {tokens} tokens, d {d}, W_g {d}x{3 * d}, W_Delta {d}x{d}, bf16",
                   "tokens": tokens, "d": d, "splits": plan["splits"], "workgroups": plan["workgroups"],
                   "weights": "row-major" if packed is None else "packed once before timing",
                   "launch": "python" if args.no_graph else "hip graph replay"},
        "roofline": roof,
        "step_tflops": round(alg["flops"] / (ms_per_step * 1e-3) / 1e12, 2),
        "step_hbm_gbs": round(alg["bytes"] / (ms_per_step * 1e-3) / 1e9, 2),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cb, parity = fusion_cpu_baseline(case, h)
        res["cpu_baseline"] = cb
        res["parity_sample"] = parity
    print(json.dumps(res), flush=True)
    fz.close()


# ---------------------------------------------------------------------------
# projected-KV cache builder (--op kvproj)
# ---------------------------------------------------------------------------

KVPROJ_METRIC = "projected-KV cache build tokens/s (L_s=3 layers, d_kv=1024, bf16) with achieved TFLOP/s and HBM GB/s"


def kvproj_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("kvproj.hip", "kvproj_common.h", "kvshot_common.h"):
        h.update(open(os.path.join(ROOT, "paper_2604_26412_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_kvproj_traffic(workload: str, kernel: str = "kvproj_kernel"):
    path = os.path.join(PROFILES, f"{kernel}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    f = re.search(r"fetch_bytes_per_launch:\s*([0-9.eE+]+)", text)
    w = re.search(r"write_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m and f and w) or m.group(1) != kvproj_source_hash():
        return None
    return float(f.group(1)) + float(w.group(1))


def make_kvproj_on_device(torch, W, spec, L=3, Hkv=8, D=128, P=16):
    """Seeded device-side generator of a projection workload: L source layer pools (N(0, 1) bf16, NaN
    spare pages) behind one random page table, W_K/W_V ~ N(0, 1/(L d_kv)), and the token list."""
    B, T, seed = spec["batch"], spec["ctx"], spec["seed"]
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    pps = T // P
    used = B * pps
    pool = used + max(1, used // 100)
    perm = torch.randperm(pool, generator=g, device="cuda")
    table = perm[:used].view(B, pps).to(torch.int32).contiguous()
    spare = perm[used:]
    pools = []
    for _ in range(2 * L):
        x = torch.randn((pool, Hkv, P, D), generator=g, device="cuda", dtype=torch.bfloat16)
        x[spare] = float("nan")
        pools.append(x)
    d_kv = Hkv * D
    sd = 1.0 / (L * d_kv) ** 0.5
    w_k = (torch.randn((d_kv, L * d_kv), generator=g, device="cuda") * sd).to(torch.bfloat16)
    w_v = (torch.randn((d_kv, L * d_kv), generator=g, device="cuda") * sd).to(torch.bfloat16)
    if spec["new"] == "all":
        counts = [T] * B
    else:
        counts = [int(c) for c in W.verify_counts(seed, B)]
    seq = torch.cat([torch.full((c,), b, dtype=torch.int32) for b, c in enumerate(counts)])
    pos = torch.cat([torch.arange(T - c, T, dtype=torch.int32) for c in counts])
    kd = torch.zeros((pool, Hkv, P, D), device="cuda", dtype=torch.bfloat16)
    vd = torch.zeros_like(kd)
    return dict(k_src=pools[:L], v_src=pools[L:], table=table, seq=seq.cuda(), pos=pos.cuda(), seq_host=seq.numpy(),
                pos_host=pos.numpy(), w_k=w_k, w_v=w_v, k_dst=kd, v_dst=vd, B=B, T=T, P=P, L=L, Hkv=Hkv, pool=pool,
                pps=pps, n=int(seq.numel()), counts=counts)


def kvproj_host_sample(torch, d, pick):
    """A compact host copy for the tokens `pick` (indices into the token list): their source pages only,
    behind a table that keeps each token's true position (the oracle rotates at it)."""
    import numpy as np

    import workloads as W

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    seq, pos, P = d["seq_host"][pick], d["pos_host"][pick], d["P"]
    keys = sorted(set(zip(seq.tolist(), (pos // P).tolist())))
    slot_of = {k: i for i, k in enumerate(keys)}
    tab_host = d["table"].cpu().numpy()
    ids = torch.tensor([int(tab_host[b, lp]) for b, lp in keys], dtype=torch.long, device="cuda")
    table = np.full((len(keys), d["pps"]), -1, np.int32)
    for (b, lp), i in slot_of.items():
        table[i, lp] = i
    cseq = np.array([slot_of[(int(b), int(p // P))] for b, p in zip(seq, pos)], np.int32)
    case = W.KvProjCase(k_src=[bits(x[ids]) for x in d["k_src"]], v_src=[bits(x[ids]) for x in d["v_src"]],
                        page_table=table, ctx_lens=np.zeros(len(keys), np.int32), token_seq=cseq,
                        token_pos=pos.astype(np.int32), w_k=bits(d["w_k"]), w_v=bits(d["w_v"]), page_size=P)
    dst = [bits(x[ids]) for x in (d["k_dst"], d["v_dst"])]
    return case, dst


def kvproj_cpu_baseline(torch, d, rope, budget_s=12.0):
    """Time the float64 projection oracle on whole sampled pages of the workload; compare the GPU cache there."""
    import numpy as np

    import oracle

    rng = np.random.default_rng(7)
    n, P = d["n"], d["P"]
    if n <= 4096:
        pick = np.arange(n)
    else:   # whole pages: 16 consecutive tokens of a random page of a random sequence
        starts = rng.choice(n // P, size=min(24576, n // P), replace=False) * P
        pick = (starts[:, None] + np.arange(P)[None, :]).ravel()
    case, dst = kvproj_host_sample(torch, d, pick)
    w_k = oracle.decode(case.w_k, "bf16")
    w_v = oracle.decode(case.w_v, "bf16")
    # timed: the oracle on growing batches of the sample until the budget is used; each batch is
    # compared with the GPU cache at once (running maxima and sums), outside the timing
    done, secs, m = 0, 0.0, min(64, case.n_tokens)
    max_abs = bound = 0.0
    sq_diff = sq_ref = 0.0
    while done < case.n_tokens and secs < budget_s:
        sl = slice(done, min(case.n_tokens, done + m))
        t0 = time.perf_counter()
        k, v = oracle.project_kv(case.k_src, case.v_src, case.page_table, case.token_seq[sl], case.token_pos[sl],
                                 w_k, w_v, page_size=P, theta=case.rope_theta, rope_keys=rope, w_dtype=None)
        secs += time.perf_counter() - t0
        pid, slot = case.token_seq[sl], case.token_pos[sl] % P
        for ref, pool in ((k, dst[0]), (v, dst[1])):
            diff = oracle.decode(pool[pid, :, slot, :], "bf16") - ref
            max_abs = max(max_abs, float(np.abs(diff).max()))
            bound = max(bound, float((np.abs(diff) / (2.0 ** -8 * np.abs(ref) + 1e-3)).max()))
            sq_diff += float((diff * diff).sum())
            sq_ref += float((ref * ref).sum())
        done = sl.stop
        m = min(2 * m, 16384)
    parity = dict(max_abs=max_abs, rel_l2=(sq_diff / sq_ref) ** 0.5, elementwise_bound_frac=bound, tokens=int(done))
    return dict(value=round(done / secs, 1), unit="tokens/s", cores=blas_threads(), kind="oracle",
                host_cpus=os.cpu_count(), seconds=round(secs, 3),
                sample=f"{done} tokens of the same workload ({'all listed tokens' if n <= 4096 else 'whole pages of random sequences'}), "
                       f"float64 NumPy oracle (weights decoded once, outside the timing)"), parity


def bench_kvproj(args, torch, K, W):
    name = args.workload or "kvproj_prefill_b64_t32k"
    if name not in W.KVPROJ_WORKLOADS:
        raise SystemExit(f"--op kvproj takes one of {sorted(W.KVPROJ_WORKLOADS)}")
    spec = W.KVPROJ_WORKLOADS[name]
    log(f"generating {name} on the device")
    d = make_kvproj_on_device(torch, W, spec)
    torch.cuda.synchronize()
    n, L, Hkv, P = d["n"], d["L"], d["Hkv"], d["P"]
    rope = not args.no_rope
    proj = K.KvProjection(num_kv_heads=Hkv, num_layers=L, page_size=P, max_pages_per_seq=d["pps"],
                          num_pages=d["pool"], max_tokens=n, max_position=d["pps"] * P)
    if args.splits:
        proj.set_option(K.OPT_SPLITS, args.splits)
    if args.kvproj_path:
        proj.set_option(K.OPT_PATH, args.kvproj_path)
    plan = proj.plan(n)

    def step():
        proj(d["k_src"], d["v_src"], d["table"], d["seq"], d["pos"], d["w_k"], d["w_v"], d["k_dst"], d["v_dst"],
             rope=rope)

    copy_calibration(torch, args.copy_calib_gib)

    log(f"{n} tokens; plan {plan}; warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run_step = step
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run_step = graph.replay
        for _ in range(min(args.warmup, 3)):
            run_step()
        torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        run_step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps
    proj.set_option(K.OPT_PROFILE, 1)
    for _ in range(args.steps):
        step()
    prof = proj.profile_read()
    proj.set_option(K.OPT_PROFILE, 0)
    calls = max(1, prof["calls"])
    main_ms, comb_ms = prof["main_ms"] / calls, prof["combine_ms"] / calls
    log(f"step {ms_per_step:.4f} ms; projection kernel {main_ms:.4f} ms; combine {comb_ms:.4f} ms")

    d_kv = Hkv * 128
    alg = W.kvproj_algorithmic(n, L, d_kv)
    part_bytes = plan["splits"] * n * 2 * d_kv * 4 if plan["splits"] > 1 else 0
    # main kernel: source vectors and weights in; the projected cache (one split) or the split partials out
    main_bytes = alg["src"] + alg["weights"] + (part_bytes if part_bytes else alg["out"])
    intensity = alg["flops"] / alg["bytes"]
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    tflops = alg["flops"] / (main_ms * 1e-3) / 1e12
    gbs = main_bytes / (main_ms * 1e-3) / 1e9
    if intensity >= ridge:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    add_mfma_ceiling(torch, K, roof)
    kfile = "kvproj_direct_kernel" if plan["path"] == 2 else "kvproj_kernel"
    roof["traffic"] = read_kvproj_traffic(name, kfile) if not (args.splits or args.no_rope or args.kvproj_path) else None
    if plan["path"] == 2:
        kname = f"kvproj_direct_kernel ({plan['tile_tokens']}-token tiles, {plan['workgroups']} workgroups)"
    else:
        kname = f"kvproj_kernel ({plan['splits']} reduction split(s), {plan['workgroups']} workgroups)"
    roof.update({"kernel": kname,
                 "kernel_ms": round(main_ms, 5), "combine_ms": round(comb_ms, 5),
                 "algorithmic_bytes_per_launch": main_bytes, "flops_per_launch": alg["flops"],
                 "arithmetic_intensity_flop_per_byte": round(intensity, 1),
                 "achieved_tflops": round(tflops, 2), "achieved_gbs": round(gbs, 2)})
    res = {
        "metric": KVPROJ_METRIC,
        "value": round(n / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{name}: {d['B']} sequences x {d['T']} tokens cached, {n} tokens projected, "
                               f"L_s {L}, d_kv {d_kv}, pages of {P}, random page table, bf16",
                   "tokens": n, "layers": L, "d_kv": d_kv, "rope": rope, "path": plan["path"],
                   "tile_tokens": plan["tile_tokens"], "splits": plan["splits"],
                   "workgroups": plan["workgroups"], "launch": "python" if args.no_graph else "hip graph replay"},
        "roofline": roof,
        "step_tflops": round(alg["flops"] / (ms_per_step * 1e-3) / 1e12, 2),
        "step_hbm_gbs": round(alg["bytes"] / (ms_per_step * 1e-3) / 1e9, 2),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cb, parity = kvproj_cpu_baseline(torch, d, rope)
        res["cpu_baseline"] = cb
        res["parity_sample"] = parity
    print(json.dumps(res), flush=True)
    proj.close()


# ---------------------------------------------------------------------------
# drafting metrics (--op accept)
# ---------------------------------------------------------------------------

ACCEPT_METRIC = "acceptance statistics (counts, step-wise rates, MAT) over verification records: records/s"


def bench_accept(args, torch, K, W):
    import numpy as np

    name = args.workload or "accept_n64m_k7"
    if name not in W.ACCEPT_WORKLOADS:
        raise SystemExit(f"--op accept takes one of {sorted(W.ACCEPT_WORKLOADS)}")
    spec = W.ACCEPT_WORKLOADS[name]
    n, steps_k = spec["n"], spec["K"]
    g = torch.Generator(device="cuda")
    g.manual_seed(spec["seed"])
    acc = torch.zeros((n,), dtype=torch.int32, device="cuda")
    alive = torch.ones((n,), dtype=torch.bool, device="cuda")
    for a in spec["rates"]:
        alive &= torch.rand((n,), generator=g, device="cuda") < a
        acc += alive.to(torch.int32)
    del alive
    torch.cuda.synchronize()
    log(f"{name}: {n} records, K = {steps_k}")

    counts = torch.empty((steps_k + 1,), dtype=torch.int64, device="cuda")
    alpha = torch.empty((steps_k,), dtype=torch.float64, device="cuda")
    mat = torch.empty((1,), dtype=torch.float64, device="cuda")
    ret = torch.empty((1,), dtype=torch.float64, device="cuda")
    lib = K.load_library()

    def step():
        st = lib.kvshot_acceptance_stats(acc.data_ptr(), n, steps_k, counts.data_ptr(), alpha.data_ptr(),
                                         mat.data_ptr(), ret.data_ptr(), 6,
                                         torch.cuda.current_stream().cuda_stream)
        if st != 0:
            raise RuntimeError(f"kvshot_acceptance_stats failed: {st}")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run_step = step
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run_step = graph.replay
        for _ in range(args.warmup):
            run_step()
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        run_step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    nbytes = 4 * n
    achieved = nbytes / (ms * 1e-3) / 1e9
    log(f"step {ms:.4f} ms; MAT {float(mat.cpu()[0]):.4f}")
    res = {
        "metric": ACCEPT_METRIC,
        "value": round(n / (ms * 1e-3), 1),
        "unit": "records/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": f"{name}: {n} accepted lengths (int32), K {steps_k}, a Markov chain with the "
                               f"gated-KV (checkpoint) step-wise rates", "records": n, "K": steps_k,
                   "launch": "python" if args.no_graph else "hip graph replay"},
        # the three launches of one call (fill, histogram, finish) are timed together: the histogram's
        # own share is at least this rate
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                     "kernel": "packed_histogram_kernel (+ fill and finish launches, timed together)",
                     "algorithmic_bytes_per_launch": nbytes},
        "result": {"mat": float(mat.cpu()[0]), "retention": float(ret.cpu()[0]),
                   "alpha": [round(float(x), 6) for x in alpha.cpu()]},
    }
    if not args.no_cpu_baseline:
        import oracle
        host = acc.cpu().numpy()
        t0 = time.perf_counter()
        rc = oracle.acceptance_counts(host, steps_k)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(n / dt, 1), "unit": "records/s", "cores": 1, "kind": "oracle",
                               "host_cpus": os.cpu_count(), "seconds": round(dt, 3),
                               "sample": f"all {n} records, NumPy counting (one thread)"}
        res["parity_sample"] = {"counts_equal": bool(np.array_equal(rc, counts.cpu().numpy())),
                                "mat_abs_diff": abs(float(mat.cpu()[0]) -
                                                    oracle.mat_from_alphas(oracle.acceptance_rates(rc)))}
    print(json.dumps(res), flush=True)


# ---------------------------------------------------------------------------
# draft-tree growth (--op treegrow)
# ---------------------------------------------------------------------------

TREEGROW_METRIC = "level-wise draft-tree growth (depth 8, top-k 10, 60 nodes) from bf16 logits: trees/s"


def treegrow_source_hash() -> str:
    h = hashlib.sha256()
    h.update(open(os.path.join(ROOT, "paper_2604_26412_amd", "csrc", "tree_grow.hip"), "rb").read())
    h.update(open(os.path.join(ROOT, "include", "kvshot_tree.h"), "rb").read())
    return h.hexdigest()[:16]


def read_treegrow_traffic(workload: str):
    """HBM bytes of one 80-row level launch from a committed counter summary, if it matches this source."""
    path = os.path.join(PROFILES, f"topk_chunk_kernel_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    f = re.search(r"fetch_bytes_per_launch:\s*([0-9.eE+]+)", text)
    w = re.search(r"write_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m and f and w) or m.group(1) != treegrow_source_hash():
        return None
    return float(f.group(1)) + float(w.group(1))


def capture(torch, fn):
    """A HIP graph of fn() (one eager run on a side stream first, as torch asks)."""
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        fn()
    torch.cuda.synchronize()
    return graph


def timed(torch, fn, steps):
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def bench_treegrow(args, torch, K, W):
    import numpy as np

    name = args.workload or "treegrow_b8_v152k_d8k10n60"
    if name not in W.TREEGROW_WORKLOADS:
        raise SystemExit(f"--op treegrow takes one of {sorted(W.TREEGROW_WORKLOADS)}")
    spec = W.TREEGROW_WORKLOADS[name]
    B, V, depth, k, n = spec["batch"], spec["vocab"], spec["depth"], spec["k"], spec["n"]
    log(f"{name}: generating {depth} levels of logits")
    host = W.treegrow_levels(spec)
    levels = [torch.from_numpy(np.ascontiguousarray(h).view(np.int16)).view(torch.bfloat16).cuda() for h in host]
    alg = W.treegrow_algorithmic(spec)
    lib = K.load_library()
    rows = [B * (1 if d == 0 else k) for d in range(depth)]
    ws = K.tree_level_workspace(B, k, V)
    lpar = torch.empty((depth, B, k), dtype=torch.int32, device="cuda")
    ltok = torch.empty((depth, B, k), dtype=torch.int32, device="cuda")
    lsc = torch.empty((depth, B, k), dtype=torch.float32, device="cuda")
    root = torch.zeros((B, 1), dtype=torch.float32, device="cuda")
    out = [torch.empty((B, n), dtype=dt, device="cuda")
           for dt in (torch.int32, torch.int32, torch.int32, torch.float32)]

    def level(d):
        F = 1 if d == 0 else k
        sc = root if d == 0 else lsc[d - 1]
        st = lib.kvshot_tree_level(levels[d].data_ptr(), K.BF16, B, F, V, V, k, sc.data_ptr(), lpar[d].data_ptr(),
                                   ltok[d].data_ptr(), lsc[d].data_ptr(), ws.data_ptr(), ws.numel(),
                                   torch.cuda.current_stream().cuda_stream)
        if st != 0:
            raise RuntimeError(f"kvshot_tree_level failed: {st}")

    def step():
        for d in range(depth):
            level(d)
        st = lib.kvshot_tree_select(B, depth, k, n, lpar.data_ptr(), ltok.data_ptr(), lsc.data_ptr(),
                                    *[o.data_ptr() for o in out], torch.cuda.current_stream().cuda_stream)
        if st != 0:
            raise RuntimeError(f"kvshot_tree_select failed: {st}")

    copy_calibration(torch, args.copy_calib_gib)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run_step = step
    if not args.no_graph:
        run_step = capture(torch, step).replay
        for _ in range(args.warmup):
            run_step()
    ms = timed(torch, run_step, args.steps)

    # the dominant kernel: one 80-row level (chunk workgroups, the last of each sequence merging and
    # expanding), 20 launches in one graph
    reps = 20
    lvl = 1 if depth > 1 else 0
    g_lvl = capture(torch, lambda: [level(lvl) for _ in range(reps)])
    g_lvl.replay()
    top_ms = timed(torch, g_lvl.replay, max(5, args.steps // 5)) / reps
    top_bytes = rows[lvl] * V * 2 + rows[lvl] * 8 + B * k * 12
    achieved = top_bytes / (top_ms * 1e-3) / 1e9
    step_gbs = alg["bytes"] / (ms * 1e-3) / 1e9
    log(f"step {ms * 1e3:.1f} us ({step_gbs:.0f} GB/s over all levels); one level of {rows[lvl]} rows "
        f"{top_ms * 1e3:.2f} us = {achieved:.0f} GB/s")

    res = {
        "metric": TREEGROW_METRIC,
        "value": round(B / (ms * 1e-3), 1),
        "unit": "trees/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 logits, f32 scores",
        "data": "synthetic",
        "config": {"workload": f"{name}: {B} sequences, vocabulary {V}, depth {depth}, top-k {k}, {n} nodes; "
                               f"{alg['rows']} logit rows ({alg['logits'] / 1e6:.1f} MB) per tree batch",
                   "batch": B, "vocab": V, "depth": depth, "k": k, "n": n,
                   "launch": "python" if args.no_graph else "hip graph replay",
                   "step_effective_gbs": round(step_gbs, 1)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": read_treegrow_traffic(name),
                     "kernel": f"topk_chunk_kernel<bf16, level> on one level of {rows[lvl]} rows",
                     "algorithmic_bytes_per_launch": top_bytes},
    }
    if not args.no_cpu_baseline:
        import oracle
        got = [o.cpu().numpy() for o in out]
        t0 = time.perf_counter()
        done, same = 0, 0
        while done < B and (done == 0 or time.perf_counter() - t0 < 12.0):
            lv = [W.bf16_bits_to_f32(h[done]).astype(np.float64) for h in host]
            rp, rt, rd, rs = oracle.grow_tree(lv, k, n)
            same += int(np.array_equal(rp, got[0][done]) and np.array_equal(rt, got[1][done]) and
                        np.array_equal(rd, got[2][done]))
            done += 1
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(done / dt, 4), "unit": "trees/s", "cores": 1,
                               "kind": "oracle", "host_cpus": os.cpu_count(), "seconds": round(dt, 3),
                               "sample": f"{done} of the {B} sequences' trees, float64 NumPy oracle (sorts "
                                         f"run on one thread)"}
        res["parity_sample"] = {"trees_checked": done, "trees_identical": same}
    print(json.dumps(res), flush=True)

if __name__ == "__main__":
    main()
