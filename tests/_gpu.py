"""Helpers for GPU tests: upload a case, run the library, compare with the oracle."""
import numpy as np

import oracle

# Parity bars (float64 oracle vs GPU output upcast to float64).
BF16_MAX_ABS = 2e-2      # stated for bf16 inputs
BF16_REL_L2 = 5e-3
# float32 inputs, float32 output, float32 arithmetic with a float32-rounded RoPE
# table: per-element error ~ a few ulp of the scores (|s| <~ 10) -> ~1e-6.
FP32_MAX_ABS = 1e-4
FP32_REL_L2 = 2e-5


def torch():
    import torch as t
    return t


def dev_array(a: np.ndarray, dtype: str = None):
    """Host array -> device tensor (bf16 bit patterns become torch.bfloat16)."""
    t = torch()
    if a.dtype == np.uint16:
        return t.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(np.ascontiguousarray(a)).cuda()


def handle_for(case, *, max_batch=None, max_pages_per_seq=None, out_dtype=None, extra_positions=0):
    from paper_2604_26412_amd import DraftAttention
    return DraftAttention(num_q_heads=case.num_q_heads, num_kv_heads=case.num_kv_heads, head_dim=case.head_dim,
                          page_size=case.page_size, dtype=case.dtype, out_dtype=out_dtype or case.dtype,
                          max_batch=max_batch or case.batch, max_draft=case.max_draft,
                          max_pages_per_seq=max_pages_per_seq or case.max_pages_per_seq, num_pages=case.num_pages,
                          max_position=case.max_pages_per_seq * case.page_size + case.max_draft + extra_positions,
                          rope_theta=case.rope_theta, softmax_scale=case.softmax_scale)


class DevCase:
    """Device copies of a case's arrays."""

    def __init__(self, case):
        self.case = case
        self.q = dev_array(case.q)
        self.k_pages = dev_array(case.k_pages)
        self.v_pages = dev_array(case.v_pages)
        self.page_table = dev_array(case.page_table)
        self.ctx_lens = dev_array(case.ctx_lens)
        self.draft_k = dev_array(case.draft_k)
        self.draft_v = dev_array(case.draft_v)
        self.extra = dev_array(case.step_offsets if case.mode == "step" else case.parents)


def run(att, dc: DevCase, *, q=None, extra=None, want_lse=False, max_ctx=None):
    t = torch()
    c = dc.case
    q = dc.q if q is None else q
    extra = dc.extra if extra is None else extra
    lse = t.empty((q.shape[0], q.shape[1], c.num_q_heads), dtype=t.float32, device="cuda") if want_lse else None
    mc = int(c.ctx_lens.max()) if max_ctx is None else max_ctx
    fn = att.step if c.mode == "step" else att.tree
    out = fn(q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, extra, max_ctx=mc,
             lse=lse)
    t.cuda.synchronize()
    o = out.float().cpu().numpy().astype(np.float64)
    return (o, lse.cpu().numpy().astype(np.float64)) if want_lse else o


def errors(gpu: np.ndarray, ref: np.ndarray):
    d = gpu - ref
    max_abs = float(np.abs(d).max())
    rel = float(np.linalg.norm(d.ravel()) / np.linalg.norm(ref.ravel()))
    return max_abs, rel


def assert_parity(gpu, ref, dtype, what=""):
    assert np.isfinite(gpu).all(), f"{what}: non-finite GPU output"
    mx, rel = errors(gpu, ref)
    if dtype == "bf16":
        assert mx <= BF16_MAX_ABS and rel <= BF16_REL_L2, f"{what}: max_abs {mx:.3e} rel_l2 {rel:.3e}"
    else:
        assert mx <= FP32_MAX_ABS and rel <= FP32_REL_L2, f"{what}: max_abs {mx:.3e} rel_l2 {rel:.3e}"
    return mx, rel


def lse_tolerance(case):
    """Per-row bound on |lse_gpu - lse_ref| (natural log) for bf16 inputs.

    The kernel rounds the rotated, scaled query and the rotated draft keys to
    bf16 (unit roundoff u = 2^-8), so each score moves by at most
    scale * (|dq| |k| + |q| |dk|) <= 2u * scale * |q| * |k|, and the
    log-sum-exp, a weighted mean of the scores to first order, by at most
    2u * scale * |q| * max|k|.  float32 accumulation adds ~1e-5.
    """
    c = case
    B, n, Hq, D = c.q.shape
    G_ = Hq // c.num_kv_heads
    qn = np.linalg.norm(oracle.decode(c.q, c.dtype), axis=-1)                   # [B][n][Hq]
    kmax = np.zeros((B, c.num_kv_heads))
    for b in range(B):
        T = int(c.ctx_lens[b])
        kt = oracle.decode(oracle.gather_prefix(c.k_pages, c.page_table[b], T, c.page_size), c.dtype)
        kd = oracle.decode(c.draft_k[b, :c.draft_len(b)], c.dtype)
        allk = np.concatenate([kt, kd], 0)
        kmax[b] = np.linalg.norm(allk, axis=-1).max(0)
    u = 2.0 ** -8 if c.dtype == "bf16" else 2.0 ** -23
    return 2 * u * c.scale * qn * np.repeat(kmax, G_, axis=1)[:, None, :] + 1e-5


def oracle_out(case, seqs=None):
    return oracle.draft_attention(case, seqs=seqs)
