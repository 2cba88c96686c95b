"""Seeded device-side inputs for the 64 x 32768 draft-attention workload.

The workload is too large to generate on the host in a test (8.6 GB of target
K/V), so it is drawn on the GPU with a seeded torch generator.  Like the rest
of ``workloads``, this module only makes inputs and copies them; it holds none
of the attention arithmetic.  ``host_sample`` copies whole sequences back into
a compact host case (bf16 bit patterns, identity page table) so the float64
oracle sees exactly the bits the GPU read.

Recipe: values N(0, 1) in bf16 (torch's normal sampler, rounded by torch);
the page pool has ~1% spare pages, filled with NaN; the page table is a seeded
random permutation of the pool (``contiguous``: sequence b owns pages
b * T / P onward, in order); step offsets are zero, so draft keys 0..n-1 are
the ones the n queries see.
"""
from __future__ import annotations

from typing import Sequence


def long_range_on_device(torch, seed: int, B: int = 64, T: int = 32768, n: int = 8, Hq: int = 32, Hkv: int = 8,
                         D: int = 128, P: int = 16, contiguous: bool = False) -> dict:
    """Device tensors of the long-range workload, plus its static geometry."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    pps = T // P
    used = B * pps
    pool = used + max(1, used // 100)
    dev = "cuda"
    kp = torch.randn((pool, Hkv, P, D), generator=g, device=dev, dtype=torch.bfloat16)
    vp = torch.randn((pool, Hkv, P, D), generator=g, device=dev, dtype=torch.bfloat16)
    perm = torch.randperm(pool, generator=g, device=dev)
    if contiguous:
        perm = torch.arange(pool, device=dev)
    table = perm[:used].view(B, pps).to(torch.int32).contiguous()
    spare = perm[used:]
    kp[spare] = float("nan")
    vp[spare] = float("nan")
    q = torch.randn((B, n, Hq, D), generator=g, device=dev, dtype=torch.bfloat16)
    dk = torch.randn((B, n, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    dv = torch.randn((B, n, Hkv, D), generator=g, device=dev, dtype=torch.bfloat16)
    lens = torch.full((B,), T, dtype=torch.int32, device=dev)
    offs = torch.zeros((B,), dtype=torch.int32, device=dev)
    return dict(mode="step", q=q, k_pages=kp, v_pages=vp, page_table=table, ctx_lens=lens, draft_k=dk, draft_v=dv,
                extra=offs, pool=pool, pps=pps, B=B, n=n, Hq=Hq, Hkv=Hkv, D=D, P=P, max_draft=n,
                lens=[T] * B, offsets=[0] * B, dtype="bf16", host=None, theta=1e6, scale=0.0)


def host_sample(torch, d: dict, seqs: Sequence[int]):
    """Copy sequences ``seqs`` of a device workload into a compact host ``DraftCase``.

    The pages of the chosen sequences are copied in page-table order, so the
    host case's page table is the identity; every bit the GPU read for those
    sequences is preserved.
    """
    import numpy as np

    from workloads import DraftCase

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    seqs = list(seqs)
    table = d["page_table"][seqs].long()
    ns, pps = table.shape
    kp = bits(d["k_pages"][table.reshape(-1)])
    vp = bits(d["v_pages"][table.reshape(-1)])
    pt = np.arange(ns * pps, dtype=np.int32).reshape(ns, pps)
    return DraftCase(mode="step", dtype="bf16", num_q_heads=d["Hq"], num_kv_heads=d["Hkv"], head_dim=d["D"],
                     page_size=d["P"], max_draft=d["max_draft"], n_new=d["n"], q=bits(d["q"][seqs]), k_pages=kp,
                     v_pages=vp, page_table=pt, ctx_lens=np.array([d["lens"][s] for s in seqs], np.int32),
                     draft_k=bits(d["draft_k"][seqs]), draft_v=bits(d["draft_v"][seqs]),
                     step_offsets=np.array([d["offsets"][s] for s in seqs], np.int32))
