#!/usr/bin/env python3
"""Benchmark of draft-step attention over reused target KV on one MI355X.

Default workload: batch 64, target context 32768, 32 query / 8 KV heads,
head_dim 128, k = 8 draft steps folded into one call, bf16, 16-token pages
with a random page table.  One "step" is one call of the library (the
attention kernel plus, with split-K, the combine kernel) over that batch.

Prints one JSON line: effective HBM GB/s (algorithmic bytes / step time),
draft tokens/s, the roofline of the dominant (attention) kernel, and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("attn_mfma.hip", "kvshot_common.h"):
        h.update(open(os.path.join(ROOT, "paper_2604_26412_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(workload: str, mode: str):
    """HBM bytes per attention launch from a committed counter summary, if it matches this kernel source."""
    path = os.path.join(PROFILES, f"attn_mfma_{workload}_{mode}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    f = re.search(r"fetch_bytes_per_launch:\s*([0-9.eE+]+)", text)
    w = re.search(r"write_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m and f and w) or m.group(1) != kernel_source_hash():
        return None
    return float(f.group(1)) + float(w.group(1))


def make_long_range_on_device(torch, seed, B=64, T=32768, n=8, Hq=32, Hkv=8, D=128, P=16):
    """Seeded device-side generator for the 64 x 32768 workload (values N(0,1), bf16)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    pps = T // P
    used = B * pps
    pool = used + max(1, used // 100)
    dev = "cuda"
    kp = torch.randn((pool, Hkv, P, D), generator=g, device=dev, dtype=torch.bfloat16)
    vp = torch.randn((pool, Hkv, P, D), generator=g, device=dev, dtype=torch.bfloat16)
    perm = torch.randperm(pool, generator=g, device=dev)
    table = perm[:used].view(B, pps).to(torch.int32).contiguous()
    spare = perm[used:]
    kp[spare] = float("nan")
    vp[spare] = float("nan")
    q = torch.randn((B, n, Hq, D), generator=g, device=dev, dtype=torch.bfloat16)
    dk = torch.randn((B, n, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    dv = torch.randn((B, n, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    lens = torch.full((B,), T, dtype=torch.int32, device=dev)
    offs = torch.zeros((B,), dtype=torch.int32, device=dev)
    return dict(q=q, k_pages=kp, v_pages=vp, page_table=table, ctx_lens=lens, draft_k=dk, draft_v=dv,
                extra=offs, pool=pool, pps=pps, B=B, T=T, n=n, Hq=Hq, Hkv=Hkv, D=D, P=P)


def host_sample(torch, d, seqs):
    """Copy sequences `seqs` of a device workload into a compact host case (for the oracle)."""
    import numpy as np

    import workloads as W

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    table = d["page_table"][seqs].long()
    ns, pps = table.shape
    kp = bits(d["k_pages"][table.reshape(-1)])
    vp = bits(d["v_pages"][table.reshape(-1)])
    pt = np.arange(ns * pps, dtype=np.int32).reshape(ns, pps)
    return W.DraftCase(mode="step", dtype="bf16", num_q_heads=d["Hq"], num_kv_heads=d["Hkv"], head_dim=d["D"],
                       page_size=d["P"], max_draft=d["n"], n_new=d["n"], q=bits(d["q"][seqs]), k_pages=kp,
                       v_pages=vp, page_table=pt, ctx_lens=np.full(ns, d["T"], np.int32),
                       draft_k=bits(d["draft_k"][seqs]), draft_v=bits(d["draft_v"][seqs]),
                       step_offsets=np.zeros(ns, np.int32))


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return int(os.environ.get("OMP_NUM_THREADS", "1"))


def cpu_baseline(torch, d, out_gpu, budget_s=15.0):
    """Time the float64 oracle on a bounded sample of whole sequences of the same workload."""
    import numpy as np

    import oracle

    first = host_sample(torch, d, [0])
    t0 = time.perf_counter()
    ref0, _ = oracle.draft_attention(first)
    t1 = time.perf_counter() - t0
    ns = int(max(1, min(8, budget_s // max(t1, 1e-3))))
    seqs = list(range(1, 1 + ns))
    case = host_sample(torch, d, seqs)
    t0 = time.perf_counter()
    ref, _ = oracle.draft_attention(case)
    dt = time.perf_counter() - t0
    per_seq_bytes = 2 * d["T"] * d["Hkv"] * d["D"] * 2 + 2 * d["n"] * d["Hkv"] * d["D"] * 2 + \
        (d["T"] // d["P"]) * 4 + 2 * d["n"] * d["Hq"] * d["D"] * 2
    got = out_gpu[[0] + seqs].float().cpu().numpy().astype(np.float64)
    allref = np.concatenate([ref0, ref], 0)
    diff = got - allref
    parity = dict(max_abs=float(np.abs(diff).max()),
                  rel_l2=float(np.linalg.norm(diff) / np.linalg.norm(allref)), sequences=1 + ns)
    return dict(value=round(ns * per_seq_bytes / dt / 1e9, 4), unit="GB/s",
                draft_tokens_per_s=round(ns * d["n"] / dt, 2), cores=blas_threads(), kind="oracle",
                host_cpus=os.cpu_count(), seconds=round(dt, 3),
                sample=f"{ns} whole sequence(s) (ctx {d['T']}, {d['n']} draft queries x {d['Hq']} heads) of the "
                       f"same workload, float64 NumPy oracle"), parity


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--mode", choices=["folded", "sequential"], default="folded")
    ap.add_argument("--splits", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=1004)
    ap.add_argument("--copy-calib-gib", type=float, default=0.0,
                    help="also run one plain device copy of this many GiB (counter calibration under a profiler)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2604_26412_amd import DraftAttention, OPT_PROFILE, OPT_SPLITS
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    log("generating the 64 x 32768 workload on the device")
    d = make_long_range_on_device(torch, args.seed)
    torch.cuda.synchronize()
    B, T, n, Hq, Hkv, D, P = d["B"], d["T"], d["n"], d["Hq"], d["Hkv"], d["D"], d["P"]
    att = DraftAttention(num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, page_size=P, dtype="bf16", max_batch=B,
                         max_draft=n, max_pages_per_seq=d["pps"], num_pages=d["pool"])
    if args.splits:
        att.set_option(OPT_SPLITS, args.splits)
    plan = att.plan(B, n if args.mode == "folded" else 1, T)
    out = torch.empty((B, n, Hq, D), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    if args.mode == "folded":
        def step():
            att.step(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["ctx_lens"], d["draft_k"], d["draft_v"],
                     d["extra"], max_ctx=T, out=out)
        queries_per_step = B * n
        calls_per_step = 1
    else:
        qs = [d["q"][:, j:j + 1].contiguous() for j in range(n)]
        offs = [torch.full((B,), j, dtype=torch.int32, device="cuda") for j in range(n)]
        outs = [torch.empty((B, 1, Hq, D), dtype=torch.bfloat16, device="cuda") for _ in range(n)]

        def step():
            for j in range(n):
                att.step(qs[j], d["k_pages"], d["v_pages"], d["page_table"], d["ctx_lens"], d["draft_k"],
                         d["draft_v"], offs[j], max_ctx=T, out=outs[j])
        queries_per_step = B * n
        calls_per_step = n

    if args.copy_calib_gib > 0:
        nbytes = int(args.copy_calib_gib * (1 << 30))
        src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {nbytes} bytes read and written by one copy kernel")
        del src, dst
    log(f"plan {plan}; warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps

    # per-kernel durations from HIP events the library records around each launch on this stream
    att.set_option(OPT_PROFILE, 1)
    for _ in range(args.steps):
        step()
    prof = att.profile_read()
    att.set_option(OPT_PROFILE, 0)
    attn_ms = prof["attn_ms"] / max(1, prof["calls"])
    comb_ms = prof["combine_ms"] / max(1, prof["calls"])
    log(f"step {ms_per_step:.4f} ms; attention kernel {attn_ms:.4f} ms; combine {comb_ms:.4f} ms")

    nq_call = n if args.mode == "folded" else 1
    # bytes one call must move: target K/V and page table once, q, the draft K/V rows it can see, out
    kv_bytes = 2 * B * T * Hkv * D * 2 + B * (T // P) * 4
    q_bytes = B * nq_call * Hq * D * 2
    out_bytes = B * nq_call * Hq * D * 2
    if args.mode == "folded":
        dkv = [2 * B * n * Hkv * D * 2]
    else:
        dkv = [2 * B * (j + 1) * Hkv * D * 2 for j in range(n)]
    step_bytes = sum(kv_bytes + q_bytes + x + out_bytes for x in dkv)
    # the attention kernel of the last call of a step (the dominant kernel; the combine writes out when split)
    attn_launch_bytes = kv_bytes + q_bytes + dkv[-1] + (out_bytes if plan["splits"] == 1 else 0)
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    achieved = attn_launch_bytes / (attn_ms * 1e-3) / 1e9
    traffic = read_traffic("long_b64_ctx32k_k8", args.mode)

    res = {
        "metric": "draft-attention effective HBM GB/s (% of peak) + draft tokens/s at 32K ctx",
        "value": round(value, 2),
        "unit": "GB/s",
        "pct_of_peak": round(100.0 * value / PEAK_HBM_GBS, 2),
        "draft_tokens_per_s": round(queries_per_step / (ms_per_step * 1e-3), 1),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"long-range draft attention: batch {B}, ctx {T}, {Hq}/{Hkv} heads, head_dim {D}, "
                               f"k={n} draft steps ({args.mode}), bf16, 16-token pages, random page table",
                   "batch": B, "ctx_len": T, "draft_steps": n, "mode": args.mode, "page_size": P,
                   "splits": plan["splits"], "workgroups": plan["workgroups"]},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": traffic, "kernel": "attn_mfma_kernel<1,4>", "kernel_ms": round(attn_ms, 5),
                     "combine_ms": round(comb_ms, 5), "algorithmic_bytes_per_launch": attn_launch_bytes},
        "whole_job_algorithmic_bytes": step_bytes,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        if args.mode == "folded":
            cb, parity = cpu_baseline(torch, d, out)
            res["cpu_baseline"] = cb
            res["parity_sample"] = parity
    print(json.dumps(res), flush=True)
    att.close()


if __name__ == "__main__":
    main()
