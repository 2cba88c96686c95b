"""Draft-step attention over reused target KV on MI355X (gfx950): Python binding.

Thin ctypes layer over ``libkvshot_draft_attn.so`` (C ABI in
``include/kvshot_draft_attn.h``).  It only marshals arguments: it checks
tensor dtypes, shapes, devices and contiguity, takes ``data_ptr()`` and the
current HIP stream from PyTorch, and calls the library.  Every step of the
computation runs in the library's HIP kernels; there is no fallback.  If the
library is missing, importing works but the first use raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

__all__ = ["DraftAttention", "GatedDeltaFusion", "KvProjection", "KvshotError", "acceptance_stats", "topk_logprobs",
           "tree_expand", "tree_select", "grow_tree", "load_library", "LIB_PATH", "EXPORTED_SYMBOLS"]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvshot_draft_attn.so")

KVSHOT_OK = 0
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "UNSUPPORTED", 3: "OUT_OF_MEMORY", 4: "DEVICE", 5: "DATA",
                6: "SCRATCH"}
BF16, FP32 = 0, 1
OPT_SPLITS, OPT_PATH, OPT_PROFILE = 0, 1, 2

EXPORTED_SYMBOLS = [
    "kvshot_draft_attn_init", "kvshot_draft_attn_destroy", "kvshot_draft_attn_step", "kvshot_draft_attn_tree",
    "kvshot_draft_attn_validate", "kvshot_draft_attn_set_option", "kvshot_draft_attn_plan",
    "kvshot_draft_attn_profile_read", "kvshot_debug_gather_kv", "kvshot_debug_tree_mask", "kvshot_debug_stream_read",
    "kvshot_debug_mfma_rate", "kvshot_status_string", "kvshot_draft_attn_call", "kvshot_draft_attn_call_noalloc",
    "kvshot_draft_attn_validate_call",
    "kvshot_fusion_init", "kvshot_fusion_destroy", "kvshot_gated_delta_fusion", "kvshot_fusion_set_option",
    "kvshot_fusion_plan", "kvshot_fusion_profile_read", "kvshot_fusion_pack_weights",
    "kvshot_gated_delta_fusion_packed",
    "kvshot_kvproj_init", "kvshot_kvproj_destroy", "kvshot_kv_project", "kvshot_kv_project_validate",
    "kvshot_kvproj_set_option", "kvshot_kvproj_plan", "kvshot_kvproj_profile_read",
    "kvshot_acceptance_stats", "kvshot_topk_workspace_bytes", "kvshot_topk_logprobs", "kvshot_tree_expand", "kvshot_tree_select",
    "kvshot_tree_level_workspace_bytes", "kvshot_tree_level",
]
FUSION_CROSS_ONLY, FUSION_OUT_FP32 = 1, 2
KVPROJ_ROPE = 1


class KvshotConfig(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32), ("dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
        ("max_batch", ctypes.c_int32), ("max_draft", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int32), ("max_position", ctypes.c_int64), ("rope_theta", ctypes.c_double),
        ("softmax_scale", ctypes.c_float), ("reserved", ctypes.c_int32), ("page_stride", ctypes.c_int64),
        ("head_stride", ctypes.c_int64), ("slot_stride", ctypes.c_int64),
    ]


MODE_STEP, MODE_TREE = 0, 1


class KvprojConfig(ctypes.Structure):
    _fields_ = [
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("num_layers", ctypes.c_int32),
        ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32), ("num_pages", ctypes.c_int32),
        ("dst_num_pages", ctypes.c_int32), ("max_tokens", ctypes.c_int32), ("max_position", ctypes.c_int64),
        ("rope_theta", ctypes.c_double), ("page_stride", ctypes.c_int64), ("head_stride", ctypes.c_int64),
        ("slot_stride", ctypes.c_int64), ("dst_page_stride", ctypes.c_int64), ("dst_head_stride", ctypes.c_int64),
        ("dst_slot_stride", ctypes.c_int64),
    ]


class KvshotCall(ctypes.Structure):
    _fields_ = [
        ("mode", ctypes.c_int32), ("batch", ctypes.c_int32), ("n_queries", ctypes.c_int32),
        ("n_nodes", ctypes.c_int32), ("max_ctx_len_hint", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("q", ctypes.c_void_p), ("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
        ("page_table", ctypes.c_void_p), ("ctx_lens", ctypes.c_void_p), ("draft_k", ctypes.c_void_p),
        ("draft_v", ctypes.c_void_p), ("step_offsets", ctypes.c_void_p), ("parents", ctypes.c_void_p),
        ("query_nodes", ctypes.c_void_p), ("pos_base", ctypes.c_void_p), ("out", ctypes.c_void_p),
        ("lse", ctypes.c_void_p),
    ]


class KvshotError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {STATUS_NAMES.get(status, status)} ({status})")
        self.status = status


_lib = None
_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64


def load_library(path: Optional[str] = None):
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2604_26412_amd.build`")
    lib = ctypes.CDLL(p)
    sig = {
        "kvshot_draft_attn_init": [ctypes.POINTER(KvshotConfig), ctypes.POINTER(_vp)],
        "kvshot_draft_attn_destroy": [_vp],
        "kvshot_draft_attn_step": [_vp, _i32, _i32, _i32] + [_vp] * 10 + [_vp],
        "kvshot_draft_attn_tree": [_vp, _i32, _i32, _i32] + [_vp] * 10 + [_vp],
        "kvshot_draft_attn_validate": [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, ctypes.POINTER(_i32), _vp],
        "kvshot_draft_attn_set_option": [_vp, _i32, _i64],
        "kvshot_draft_attn_plan": [_vp, _i32, _i32, _i32] + [ctypes.POINTER(_i32)] * 4,
        "kvshot_draft_attn_profile_read": [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(_i64)],
        "kvshot_debug_gather_kv": [_vp, _i32, _i32] + [_vp] * 7,
        "kvshot_debug_tree_mask": [_vp, _i32, _i32, _vp, _vp, _vp, _vp],
        "kvshot_debug_stream_read": [_vp, _i64, _vp, _i32, _vp],
        "kvshot_debug_mfma_rate": [_i32, _i32, _vp, _vp],
        "kvshot_draft_attn_call": [_vp, ctypes.POINTER(KvshotCall), _vp],
        "kvshot_draft_attn_call_noalloc": [_vp, ctypes.POINTER(KvshotCall), _vp],
        "kvshot_draft_attn_validate_call": [_vp, ctypes.POINTER(KvshotCall), ctypes.POINTER(_i32), _vp],
        "kvshot_fusion_init": [_i32, _i32, ctypes.POINTER(_vp)],
        "kvshot_fusion_destroy": [_vp],
        "kvshot_gated_delta_fusion": [_vp, _i32] + [_vp] * 7 + [_i32, _vp],
        "kvshot_fusion_set_option": [_vp, _i32, _i64],
        "kvshot_fusion_pack_weights": [_vp, _vp, _vp, _vp, _vp],
        "kvshot_gated_delta_fusion_packed": [_vp, _i32] + [_vp] * 6 + [_i32, _vp],
        "kvshot_fusion_plan": [_vp, _i32, ctypes.POINTER(_i32), ctypes.POINTER(_i32)],
        "kvshot_fusion_profile_read": [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(_i64)],
        "kvshot_kvproj_init": [ctypes.POINTER(KvprojConfig), ctypes.POINTER(_vp)],
        "kvshot_kvproj_destroy": [_vp],
        "kvshot_kv_project": [_vp, _i32, _i32, ctypes.POINTER(_vp), ctypes.POINTER(_vp)] + [_vp] * 8 + [_i32, _vp],
        "kvshot_kv_project_validate": [_vp, _i32, _i32, _vp, _vp, _vp, _vp, ctypes.POINTER(_i32),
                                       ctypes.POINTER(_i32), _vp],
        "kvshot_kvproj_set_option": [_vp, _i32, _i64],
        "kvshot_kvproj_plan": [_vp, _i32, ctypes.POINTER(_i32), ctypes.POINTER(_i32), ctypes.POINTER(_i32),
                               ctypes.POINTER(_i32)],
        "kvshot_kvproj_profile_read": [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(_i64)],
        "kvshot_acceptance_stats": [_vp, _i64, _i32, _vp, _vp, _vp, _vp, _i32, _vp],
        "kvshot_topk_logprobs": [_vp, _i32, _i32, _i32, _i64, _i32, _vp, _vp, _vp, _i64, _vp],
        "kvshot_tree_expand": [_i32, _i32, _i32, _i32] + [_vp] * 6 + [_vp],
        "kvshot_tree_select": [_i32, _i32, _i32, _i32] + [_vp] * 7 + [_vp],
        "kvshot_tree_level": [_vp, _i32, _i32, _i32, _i32, _i64, _i32] + [_vp] * 5 + [_i64, _vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.kvshot_topk_workspace_bytes.argtypes = [_i32, _i32]
    lib.kvshot_topk_workspace_bytes.restype = _i64
    lib.kvshot_tree_level_workspace_bytes.argtypes = [_i32, _i32, _i32]
    lib.kvshot_tree_level_workspace_bytes.restype = _i64
    lib.kvshot_status_string.argtypes = [_i32]
    lib.kvshot_status_string.restype = ctypes.c_char_p
    if path is None:
        _lib = lib
    return lib


def _check(fn: str, status: int):
    if status != KVSHOT_OK:
        raise KvshotError(fn, status)


def _torch():
    import torch
    return torch


def _dtype_code(name: str) -> int:
    if name in ("bf16", "bfloat16"):
        return BF16
    if name in ("fp32", "float32"):
        return FP32
    raise ValueError(f"dtype must be bf16 or fp32, got {name!r}")


def stream_read(src, sink=None, workgroups: int = 2048, stream=None):
    """Read every byte of device tensor `src` once (streaming-read bandwidth probe)."""
    torch = _torch()
    lib = load_library()
    if sink is None:
        sink = torch.empty(workgroups * 4, dtype=torch.int32, device=src.device)
    st = lib.kvshot_debug_stream_read(src.data_ptr(), src.numel() * src.element_size(), sink.data_ptr(), workgroups,
                                      stream if stream is not None else torch.cuda.current_stream().cuda_stream)
    _check("kvshot_debug_stream_read", st)
    return sink


def mfma_rate(iters: int, workgroups: int = 256, sink=None, stream=None):
    """Dense bf16 matrix work with no memory traffic (matrix-rate probe); returns the sink.
    One launch performs workgroups x 4 x iters x 16 x 32768 flops."""
    torch = _torch()
    lib = load_library()
    if sink is None:
        sink = torch.empty(workgroups * 4, dtype=torch.int32, device="cuda")
    st = lib.kvshot_debug_mfma_rate(workgroups, iters, sink.data_ptr(),
                                    stream if stream is not None else torch.cuda.current_stream().cuda_stream)
    _check("kvshot_debug_mfma_rate", st)
    return sink


class DraftAttention:
    """One configured handle of the library (see ``kvshot_config`` in the header)."""

    def __init__(self, *, num_q_heads: int = 32, num_kv_heads: int = 8, head_dim: int = 128, page_size: int = 16,
                 dtype: str = "bf16", out_dtype: Optional[str] = None, max_batch: int, max_draft: int,
                 max_pages_per_seq: int, num_pages: int, max_position: Optional[int] = None,
                 rope_theta: float = 1e6, softmax_scale: float = 0.0, page_stride: int = 0, head_stride: int = 0,
                 slot_stride: int = 0):
        self._lib = load_library()
        cfg = KvshotConfig()
        cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim = num_q_heads, num_kv_heads, head_dim
        cfg.page_size = page_size
        cfg.dtype = _dtype_code(dtype)
        cfg.out_dtype = _dtype_code(out_dtype or dtype)
        cfg.max_batch, cfg.max_draft = max_batch, max_draft
        cfg.max_pages_per_seq, cfg.num_pages = max_pages_per_seq, num_pages
        cfg.max_position = max_position if max_position is not None else max_pages_per_seq * page_size + max_draft
        cfg.rope_theta, cfg.softmax_scale, cfg.reserved = rope_theta, softmax_scale, 0
        cfg.page_stride, cfg.head_stride, cfg.slot_stride = page_stride, head_stride, slot_stride
        self.cfg = cfg
        self.dtype = dtype
        self.out_dtype = out_dtype or dtype
        h = _vp()
        _check("kvshot_draft_attn_init", self._lib.kvshot_draft_attn_init(ctypes.byref(cfg), ctypes.byref(h)))
        self._h = h

    # -- lifetime ---------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self._lib.kvshot_draft_attn_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # -- argument marshalling ----------------------------------------------
    def _elem_dtype(self):
        torch = _torch()
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def _tensor(self, t, name, dtype, shape=None, ndim=None):
        torch = _torch()
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU")
        if dtype is not None and t.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if shape is not None and tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        if ndim is not None and t.dim() != ndim:
            raise ValueError(f"{name} must have {ndim} dims")
        return t.data_ptr()

    def _common(self, q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, out, lse):
        torch = _torch()
        c = self.cfg
        ed = self._elem_dtype()
        B, n = q.shape[0], q.shape[1]
        D, Hq, Hkv = c.head_dim, c.num_q_heads, c.num_kv_heads
        ptrs = dict(
            q=self._tensor(q, "q", ed, (B, n, Hq, D)),
            k=self._tensor(k_pages, "k_pages", ed),
            v=self._tensor(v_pages, "v_pages", ed),
            pt=self._tensor(page_table, "page_table", torch.int32, (B, c.max_pages_per_seq)),
            lens=self._tensor(ctx_lens, "ctx_lens", torch.int32, (B,)),
            dk=self._tensor(draft_k, "draft_k", ed, (B, c.max_draft, Hkv, D)),
            dv=self._tensor(draft_v, "draft_v", ed, (B, c.max_draft, Hkv, D)),
        )
        if k_pages.numel() < c.num_pages * (c.page_stride or Hkv * c.page_size * D):
            raise ValueError("k_pages smaller than num_pages pages")
        if v_pages.numel() < c.num_pages * (c.page_stride or Hkv * c.page_size * D):
            raise ValueError("v_pages smaller than num_pages pages")
        od = torch.bfloat16 if self.out_dtype == "bf16" else torch.float32
        if out is None:
            out = torch.empty((B, n, Hq, D), dtype=od, device=q.device)
        ptrs["out"] = self._tensor(out, "out", od, (B, n, Hq, D))
        ptrs["lse"] = self._tensor(lse, "lse", torch.float32, (B, n, Hq)) if lse is not None else None
        return ptrs, out

    @staticmethod
    def _stream(stream):
        if stream is not None:
            return stream
        return _torch().cuda.current_stream().cuda_stream

    def _hint(self, max_ctx):
        return self.cfg.max_pages_per_seq * self.cfg.page_size if max_ctx is None else int(max_ctx)

    # -- calls -------------------------------------------------------------
    def step(self, q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, step_offsets, *, max_ctx=None,
             out=None, lse=None, pos_base=None, stream=None, noalloc=False):
        """Causal draft steps; returns ``out`` [B][n_new][Hq][D].

        ``pos_base`` (int32 [B]) places draft step 0 of sequence b at position pos_base[b] instead of
        ctx_lens[b] (see ``kvshot_call`` in the header).  ``noalloc`` calls
        ``kvshot_draft_attn_call_noalloc`` (split partials in the library's static scratch).
        """
        torch = _torch()
        ptrs, out = self._common(q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, out, lse)
        B = q.shape[0]
        offs = self._tensor(step_offsets, "step_offsets", torch.int32, (B,))
        if pos_base is None and not noalloc:
            _check("kvshot_draft_attn_step", self._lib.kvshot_draft_attn_step(
                self._h, B, q.shape[1], self._hint(max_ctx), ptrs["q"], ptrs["k"], ptrs["v"], ptrs["pt"],
                ptrs["lens"], ptrs["dk"], ptrs["dv"], offs, ptrs["out"], ptrs["lse"], self._stream(stream)))
            return out
        call = self._call(MODE_STEP, q, q.shape[1], 0, max_ctx, ptrs, pos_base)
        call.step_offsets = offs
        self._run_call(call, stream, noalloc)
        return out

    def _run_call(self, call, stream, noalloc):
        name = "kvshot_draft_attn_call_noalloc" if noalloc else "kvshot_draft_attn_call"
        _check(name, getattr(self._lib, name)(self._h, ctypes.byref(call), self._stream(stream)))

    def tree(self, q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, parents, *, max_ctx=None,
             out=None, lse=None, query_nodes=None, pos_base=None, stream=None, noalloc=False):
        """Draft-tree queries with an ancestor-or-self mask; returns ``out`` [B][n_queries][Hq][D].

        ``parents`` is [B][n_nodes]; without ``query_nodes`` every node has a query row (n_queries ==
        n_nodes).  ``query_nodes`` (int32 [B][n_queries]) names the node of each query row, so a tree grown
        level by level needs queries for its newest level only.  ``pos_base`` and ``noalloc`` as in
        :meth:`step`.
        """
        torch = _torch()
        ptrs, out = self._common(q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, out, lse)
        B, nq = q.shape[0], q.shape[1]
        n_nodes = parents.shape[1] if parents.dim() == 2 else -1
        par = self._tensor(parents, "parents", torch.int32, (B, n_nodes))
        if query_nodes is None and pos_base is None and not noalloc:
            if n_nodes != nq:
                raise ValueError("parents must be [B][n_queries] without query_nodes")
            _check("kvshot_draft_attn_tree", self._lib.kvshot_draft_attn_tree(
                self._h, B, nq, self._hint(max_ctx), ptrs["q"], ptrs["k"], ptrs["v"], ptrs["pt"],
                ptrs["lens"], ptrs["dk"], ptrs["dv"], par, ptrs["out"], ptrs["lse"], self._stream(stream)))
            return out
        call = self._call(MODE_TREE, q, nq, n_nodes, max_ctx, ptrs, pos_base)
        call.parents = par
        if query_nodes is not None:
            call.query_nodes = self._tensor(query_nodes, "query_nodes", torch.int32, (B, nq))
        self._run_call(call, stream, noalloc)
        return out

    def _call(self, mode, q, nq, n_nodes, max_ctx, ptrs, pos_base):
        torch = _torch()
        c = KvshotCall()
        c.mode, c.batch, c.n_queries, c.n_nodes = mode, q.shape[0], nq, n_nodes
        c.max_ctx_len_hint, c.reserved = self._hint(max_ctx), 0
        c.q, c.k_pages, c.v_pages = ptrs["q"], ptrs["k"], ptrs["v"]
        c.page_table, c.ctx_lens, c.draft_k, c.draft_v = ptrs["pt"], ptrs["lens"], ptrs["dk"], ptrs["dv"]
        c.out, c.lse = ptrs["out"], ptrs["lse"]
        if pos_base is not None:
            c.pos_base = self._tensor(pos_base, "pos_base", torch.int32, (q.shape[0],))
        return c

    def validate(self, page_table, ctx_lens, n_queries, *, step_offsets=None, parents=None, max_ctx=None,
                 stream=None):
        """Returns 0 if the device data honours the contract, else the first violation code (1..4)."""
        torch = _torch()
        B = ctx_lens.shape[0]
        pt = self._tensor(page_table, "page_table", torch.int32, (B, self.cfg.max_pages_per_seq))
        lens = self._tensor(ctx_lens, "ctx_lens", torch.int32, (B,))
        so = self._tensor(step_offsets, "step_offsets", torch.int32, (B,)) if step_offsets is not None else None
        par = self._tensor(parents, "parents", torch.int32, (B, n_queries)) if parents is not None else None
        bad = _i32(0)
        st = self._lib.kvshot_draft_attn_validate(self._h, B, n_queries, self._hint(max_ctx), pt, lens, so, par,
                                                  ctypes.byref(bad), self._stream(stream))
        if st not in (KVSHOT_OK, 5):
            raise KvshotError("kvshot_draft_attn_validate", st)
        return int(bad.value)

    def set_option(self, option: int, value: int):
        _check("kvshot_draft_attn_set_option", self._lib.kvshot_draft_attn_set_option(self._h, option, value))

    def plan(self, batch: int, n_queries: int, max_ctx: Optional[int] = None):
        vals = [_i32(0) for _ in range(4)]
        _check("kvshot_draft_attn_plan", self._lib.kvshot_draft_attn_plan(
            self._h, batch, n_queries, self._hint(max_ctx), *[ctypes.byref(v) for v in vals]))
        return dict(splits=vals[0].value, path=vals[1].value, row_tiles=vals[2].value, workgroups=vals[3].value)

    def profile_read(self):
        a, c, n = ctypes.c_double(0), ctypes.c_double(0), _i64(0)
        _check("kvshot_draft_attn_profile_read", self._lib.kvshot_draft_attn_profile_read(
            self._h, ctypes.byref(a), ctypes.byref(c), ctypes.byref(n)))
        return dict(attn_ms=a.value, combine_ms=c.value, calls=n.value)

    def debug_gather_kv(self, k_pages, v_pages, page_table, ctx_lens, max_ctx, stream=None):
        torch = _torch()
        c = self.cfg
        ed = self._elem_dtype()
        B = ctx_lens.shape[0]
        kd = torch.empty((B, max_ctx, c.num_kv_heads, c.head_dim), dtype=ed, device=k_pages.device)
        vd = torch.empty_like(kd)
        _check("kvshot_debug_gather_kv", self._lib.kvshot_debug_gather_kv(
            self._h, B, max_ctx, self._tensor(k_pages, "k_pages", ed), self._tensor(v_pages, "v_pages", ed),
            self._tensor(page_table, "page_table", torch.int32, (B, c.max_pages_per_seq)),
            self._tensor(ctx_lens, "ctx_lens", torch.int32, (B,)), kd.data_ptr(), vd.data_ptr(),
            self._stream(stream)))
        return kd, vd

    def debug_tree_mask(self, parents, stream=None):
        torch = _torch()
        B, n = parents.shape
        anc = torch.empty((B, n), dtype=torch.int64, device=parents.device)
        depth = torch.empty((B, n), dtype=torch.int32, device=parents.device)
        _check("kvshot_debug_tree_mask", self._lib.kvshot_debug_tree_mask(
            self._h, B, n, self._tensor(parents, "parents", torch.int32, (B, n)), anc.data_ptr(), depth.data_ptr(),
            self._stream(stream)))
        return anc, depth


def acceptance_stats(accepted, K: int, retention_step: Optional[int] = None, stream=None):
    """Counts c_k = #{a >= k} (int64 [K + 1]), step-wise rates alpha (float64 [K]), MAT (float64 [1]) and,
    with ``retention_step``, alpha[retention_step] / alpha[0] (float64 [1]) for the accepted draft lengths
    ``accepted`` (int32 device tensor) -- C ABI in ``include/kvshot_metrics.h``."""
    torch = _torch()
    lib = load_library()
    dev = accepted.device
    n = accepted.numel()
    acc = GatedDeltaFusion._tensor(accepted, "accepted", torch.int32, (n,)) if n else None
    counts = torch.empty((K + 1,), dtype=torch.int64, device=dev)
    alpha = torch.empty((K,), dtype=torch.float64, device=dev)
    mat = torch.empty((1,), dtype=torch.float64, device=dev)
    ret = torch.empty((1,), dtype=torch.float64, device=dev) if retention_step is not None else None
    _check("kvshot_acceptance_stats", lib.kvshot_acceptance_stats(
        acc, n, K, counts.data_ptr(), alpha.data_ptr(), mat.data_ptr(), ret.data_ptr() if ret is not None else None,
        retention_step if retention_step is not None else 0,
        stream if stream is not None else torch.cuda.current_stream().cuda_stream))
    return counts, alpha, mat, ret


def _stream_of(stream):
    return stream if stream is not None else _torch().cuda.current_stream().cuda_stream


def topk_workspace_bytes(rows: int, vocab: int) -> int:
    """Device scratch ``topk_logprobs`` needs for ``rows`` rows of ``vocab`` logits (0: none)."""
    n = load_library().kvshot_topk_workspace_bytes(int(rows), int(vocab))
    if n < 0:
        raise ValueError(f"no top-k plan for rows={rows}, vocab={vocab}")
    return int(n)


def topk_logprobs(logits, k: int, workspace=None, stream=None):
    """Top-k tokens (int32 [..., k]) and their log-softmax values (float32 [..., k]) of each row of
    ``logits`` (bf16 or float32 device tensor [..., vocab], rows contiguous) -- ``include/kvshot_tree.h``.
    ``workspace``: a device tensor of at least ``topk_workspace_bytes`` bytes, allocated here if None."""
    torch = _torch()
    lib = load_library()
    if logits.dtype not in (torch.bfloat16, torch.float32) or not logits.is_cuda or logits.stride(-1) != 1:
        raise ValueError("logits must be a bf16 or float32 device tensor with contiguous rows")
    vocab = logits.shape[-1]
    rows = logits.numel() // vocab
    flat = logits if logits.dim() == 2 else logits.reshape(rows, vocab)   # a 2-D view keeps its row stride
    need = topk_workspace_bytes(rows, vocab)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=logits.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    tokens = torch.empty(logits.shape[:-1] + (k,), dtype=torch.int32, device=logits.device)
    lp = torch.empty(logits.shape[:-1] + (k,), dtype=torch.float32, device=logits.device)
    _check("kvshot_topk_logprobs", lib.kvshot_topk_logprobs(
        flat.data_ptr(), BF16 if logits.dtype == torch.bfloat16 else FP32, rows, vocab, flat.stride(0), k,
        tokens.data_ptr(), lp.data_ptr(), ws_ptr, ws_bytes, _stream_of(stream)))
    return tokens, lp


def tree_expand(scores, tokens, logprobs, k: int, out=None, stream=None):
    """Next frontier (parent index, token, score; each [batch][k]) from the frontier's scores [batch][F] and
    proposals tokens / logprobs [batch][F][P]; ``out`` = (parent, token, score) buffers to fill."""
    torch = _torch()
    lib = load_library()
    batch, frontier, proposals = tokens.shape
    sc = GatedDeltaFusion._tensor(scores, "scores", torch.float32, (batch, frontier))
    tk = GatedDeltaFusion._tensor(tokens, "tokens", torch.int32, (batch, frontier, proposals))
    lp = GatedDeltaFusion._tensor(logprobs, "logprobs", torch.float32, (batch, frontier, proposals))
    if out is None:
        out = (torch.empty((batch, k), dtype=torch.int32, device=tokens.device),
               torch.empty((batch, k), dtype=torch.int32, device=tokens.device),
               torch.empty((batch, k), dtype=torch.float32, device=tokens.device))
    par, tok, nsc = out
    for t, name, dt in ((par, "parent", torch.int32), (tok, "token", torch.int32), (nsc, "score", torch.float32)):
        GatedDeltaFusion._tensor(t, name, dt, (batch, k))
    _check("kvshot_tree_expand", lib.kvshot_tree_expand(batch, frontier, proposals, k, sc, tk, lp, par.data_ptr(),
                                                        tok.data_ptr(), nsc.data_ptr(), _stream_of(stream)))
    return par, tok, nsc


def tree_select(level_parent, level_tokens, level_scores, n: int, stream=None):
    """The tree (parents, tokens, depths, scores; each [batch][n]) from the frontiers of every level
    ([depth][batch][k] each)."""
    torch = _torch()
    lib = load_library()
    depth, batch, k = level_tokens.shape
    lpar = GatedDeltaFusion._tensor(level_parent, "level_parent", torch.int32, (depth, batch, k))
    ltok = GatedDeltaFusion._tensor(level_tokens, "level_tokens", torch.int32, (depth, batch, k))
    lsc = GatedDeltaFusion._tensor(level_scores, "level_scores", torch.float32, (depth, batch, k))
    dev = level_tokens.device
    out = [torch.empty((batch, n), dtype=torch.int32, device=dev) for _ in range(3)]
    osc = torch.empty((batch, n), dtype=torch.float32, device=dev)
    _check("kvshot_tree_select", lib.kvshot_tree_select(batch, depth, k, n, lpar, ltok, lsc, out[0].data_ptr(),
                                                        out[1].data_ptr(), out[2].data_ptr(), osc.data_ptr(),
                                                        _stream_of(stream)))
    return out[0], out[1], out[2], osc


def tree_level_workspace(batch: int, frontier: int, vocab: int, device="cuda"):
    """A zero-filled workspace for ``tree_level`` (its counters must start at zero; calls leave them so)."""
    torch = _torch()
    n = load_library().kvshot_tree_level_workspace_bytes(int(batch), int(frontier), int(vocab))
    if n < 0:
        raise ValueError(f"no tree-level plan for batch={batch}, frontier={frontier}, vocab={vocab}")
    return torch.zeros(int(n), dtype=torch.uint8, device=device)


def tree_level(logits, scores, k: int, workspace=None, out=None, stream=None):
    """One level of growth in one launch: ``logits`` [batch][F][vocab] (bf16 or float32, rows contiguous),
    ``scores`` [batch][F] float32 -> next frontier (parent index, token, score; each [batch][k])."""
    torch = _torch()
    lib = load_library()
    if logits.dtype not in (torch.bfloat16, torch.float32) or not logits.is_cuda or logits.dim() != 3 \
            or not logits.is_contiguous():
        raise ValueError("logits must be a contiguous bf16 or float32 device tensor [batch][frontier][vocab]")
    batch, frontier, vocab = logits.shape
    sc = GatedDeltaFusion._tensor(scores, "scores", torch.float32, (batch, frontier))
    if workspace is None:
        workspace = tree_level_workspace(batch, frontier, vocab, logits.device)
    if out is None:
        out = (torch.empty((batch, k), dtype=torch.int32, device=logits.device),
               torch.empty((batch, k), dtype=torch.int32, device=logits.device),
               torch.empty((batch, k), dtype=torch.float32, device=logits.device))
    par, tok, nsc = out
    for t, name, dt in ((par, "parent", torch.int32), (tok, "token", torch.int32), (nsc, "score", torch.float32)):
        GatedDeltaFusion._tensor(t, name, dt, (batch, k))
    _check("kvshot_tree_level", lib.kvshot_tree_level(
        logits.data_ptr(), BF16 if logits.dtype == torch.bfloat16 else FP32, batch, frontier, vocab, vocab, k, sc,
        par.data_ptr(), tok.data_ptr(), nsc.data_ptr(), workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), _stream_of(stream)))
    return par, tok, nsc


def grow_tree(level_logits, k: int, n: int, stream=None):
    """Grow a tree level by level: ``level_logits[d]`` holds the drafter's logits for level d's frontier
    ([batch][1][vocab] for the root, then [batch][k][vocab], frontier nodes in the order the previous level
    returned them).  Only sequences the library calls."""
    torch = _torch()
    batch = level_logits[0].shape[0]
    dev = level_logits[0].device
    depth = len(level_logits)
    lpar = torch.empty((depth, batch, k), dtype=torch.int32, device=dev)
    ltok = torch.empty((depth, batch, k), dtype=torch.int32, device=dev)
    lsc = torch.empty((depth, batch, k), dtype=torch.float32, device=dev)
    scores = torch.zeros((batch, 1), dtype=torch.float32, device=dev)
    vocab = level_logits[0].shape[-1]
    ws = tree_level_workspace(batch, max(z.shape[1] for z in level_logits), vocab, dev)
    for d, z in enumerate(level_logits):
        tree_level(z, scores, k, workspace=ws, out=(lpar[d], ltok[d], lsc[d]), stream=stream)
        scores = lsc[d]
    return tree_select(lpar, ltok, lsc, n, stream)


class GatedDeltaFusion:
    """Handle for the hybrid drafter's gated delta fusion (C ABI in ``include/kvshot_fusion.h``).

    ``h = n + sigmoid(W_g [n; o; o - n] + b_g) * (W_Delta (o - n))`` per token,
    with bf16 activations and weights and a float32 bias.
    """

    def __init__(self, d: int, max_tokens: int):
        self._lib = load_library()
        self.d, self.max_tokens = int(d), int(max_tokens)
        h = _vp()
        _check("kvshot_fusion_init", self._lib.kvshot_fusion_init(self.d, self.max_tokens, ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self._lib.kvshot_fusion_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    @staticmethod
    def _tensor(t, name, dtype, shape):
        torch = _torch()
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU")
        if t.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        return t.data_ptr()

    def __call__(self, n, o, w_g, b_g, w_delta, *, out=None, gate=None, cross_only=False, out_dtype="bf16",
                 packed=None, stream=None):
        """Returns ``out`` [tokens][d]; ``gate`` (float32 [tokens][d]) is filled when given.

        With ``packed`` (from :meth:`pack_weights`), ``w_g`` and ``w_delta`` are not read and may be None.
        """
        torch = _torch()
        bf = torch.bfloat16
        tokens, d = o.shape[0], self.d
        od = torch.bfloat16 if out_dtype in ("bf16", "bfloat16") else torch.float32
        if out is None:
            out = torch.empty((tokens, d), dtype=od, device=o.device)
        n_ptr = None if (cross_only and n is None) else self._tensor(n, "n", bf, (tokens, d))
        flags = (FUSION_CROSS_ONLY if cross_only else 0) | (FUSION_OUT_FP32 if od == torch.float32 else 0)
        o_ptr = self._tensor(o, "o", bf, (tokens, d))
        b_ptr = self._tensor(b_g, "b_g", torch.float32, (d,))
        out_ptr = self._tensor(out, "out", od, (tokens, d))
        g_ptr = self._tensor(gate, "gate", torch.float32, (tokens, d)) if gate is not None else None
        s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
        if packed is not None:
            _check("kvshot_gated_delta_fusion_packed", self._lib.kvshot_gated_delta_fusion_packed(
                self._h, tokens, n_ptr, o_ptr, self._tensor(packed, "packed", bf, (4 * d * d,)), b_ptr, out_ptr,
                g_ptr, flags, s))
        else:
            _check("kvshot_gated_delta_fusion", self._lib.kvshot_gated_delta_fusion(
                self._h, tokens, n_ptr, o_ptr, self._tensor(w_g, "w_g", bf, (d, 3 * d)), b_ptr,
                self._tensor(w_delta, "w_delta", bf, (d, d)), out_ptr, g_ptr, flags, s))
        return out

    def pack_weights(self, w_g, w_delta, packed=None, stream=None):
        """Packed copy of both weight matrices (bf16 [4 d^2]) for ``__call__(..., packed=...)``."""
        torch = _torch()
        d = self.d
        if packed is None:
            packed = torch.empty((4 * d * d,), dtype=torch.bfloat16, device=w_g.device)
        _check("kvshot_fusion_pack_weights", self._lib.kvshot_fusion_pack_weights(
            self._h, self._tensor(w_g, "w_g", torch.bfloat16, (d, 3 * d)),
            self._tensor(w_delta, "w_delta", torch.bfloat16, (d, d)),
            self._tensor(packed, "packed", torch.bfloat16, (4 * d * d,)),
            stream if stream is not None else torch.cuda.current_stream().cuda_stream))
        return packed

    def set_option(self, option: int, value: int):
        _check("kvshot_fusion_set_option", self._lib.kvshot_fusion_set_option(self._h, option, value))

    def plan(self, tokens: int):
        s, w = _i32(0), _i32(0)
        _check("kvshot_fusion_plan", self._lib.kvshot_fusion_plan(self._h, tokens, ctypes.byref(s), ctypes.byref(w)))
        return dict(splits=s.value, workgroups=w.value)

    def profile_read(self):
        a, c, k = ctypes.c_double(0), ctypes.c_double(0), _i64(0)
        _check("kvshot_fusion_profile_read", self._lib.kvshot_fusion_profile_read(
            self._h, ctypes.byref(a), ctypes.byref(c), ctypes.byref(k)))
        return dict(main_ms=a.value, combine_ms=c.value, calls=k.value)


class KvProjection:
    """Handle for the projected-KV cache builder (C ABI in ``include/kvshot_kvproj.h``).

    For each listed token, ``k' = W_K [k^(1); ...; k^(L_s)]`` (rotated at the
    token's position with ``rope=True``) and ``v' = W_V [v^(1); ...]`` are
    written into the destination pools at the token's slot.
    """

    def __init__(self, *, num_kv_heads: int = 8, head_dim: int = 128, num_layers: int = 3, page_size: int = 16,
                 max_pages_per_seq: int, num_pages: int, dst_num_pages: Optional[int] = None, max_tokens: int,
                 max_position: int, rope_theta: float = 1e6):
        self._lib = load_library()
        self.cfg = KvprojConfig(num_kv_heads=num_kv_heads, head_dim=head_dim, num_layers=num_layers,
                                page_size=page_size, max_pages_per_seq=max_pages_per_seq, num_pages=num_pages,
                                dst_num_pages=dst_num_pages if dst_num_pages is not None else num_pages,
                                max_tokens=max_tokens, max_position=max_position, rope_theta=rope_theta)
        h = _vp()
        _check("kvshot_kvproj_init", self._lib.kvshot_kvproj_init(ctypes.byref(self.cfg), ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self._lib.kvshot_kvproj_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def _pool(self, t, name, npages):
        shape = (npages, self.cfg.num_kv_heads, self.cfg.page_size, self.cfg.head_dim)
        return GatedDeltaFusion._tensor(t, name, _torch().bfloat16, shape)

    def _tables(self, page_table, token_seq, token_pos, dst_page_table):
        torch = _torch()
        n = token_seq.shape[0]
        batch = page_table.shape[0]
        mp = self.cfg.max_pages_per_seq
        pt = GatedDeltaFusion._tensor(page_table, "page_table", torch.int32, (batch, mp))
        dpt = (GatedDeltaFusion._tensor(dst_page_table, "dst_page_table", torch.int32, (batch, mp))
               if dst_page_table is not None else None)
        ts = GatedDeltaFusion._tensor(token_seq, "token_seq", torch.int32, (n,))
        tp = GatedDeltaFusion._tensor(token_pos, "token_pos", torch.int32, (n,))
        return n, batch, pt, ts, tp, dpt

    def __call__(self, k_src, v_src, page_table, token_seq, token_pos, w_k, w_v, k_dst, v_dst, *,
                 dst_page_table=None, rope: bool = True, stream=None):
        """Projects the listed tokens into ``k_dst`` / ``v_dst`` (bf16 pools, written in place)."""
        torch = _torch()
        L = self.cfg.num_layers
        if len(k_src) != L or len(v_src) != L:
            raise ValueError(f"k_src and v_src must hold {L} pools")
        n, batch, pt, ts, tp, dpt = self._tables(page_table, token_seq, token_pos, dst_page_table)
        ks = (_vp * L)(*[self._pool(t, f"k_src[{i}]", self.cfg.num_pages) for i, t in enumerate(k_src)])
        vs = (_vp * L)(*[self._pool(t, f"v_src[{i}]", self.cfg.num_pages) for i, t in enumerate(v_src)])
        d_kv = self.cfg.num_kv_heads * self.cfg.head_dim
        wk = GatedDeltaFusion._tensor(w_k, "w_k", torch.bfloat16, (d_kv, L * d_kv))
        wv = GatedDeltaFusion._tensor(w_v, "w_v", torch.bfloat16, (d_kv, L * d_kv))
        kd = self._pool(k_dst, "k_dst", self.cfg.dst_num_pages)
        vd = self._pool(v_dst, "v_dst", self.cfg.dst_num_pages)
        s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
        _check("kvshot_kv_project", self._lib.kvshot_kv_project(
            self._h, n, batch, ks, vs, pt, ts, tp, wk, wv, kd, vd, dpt, KVPROJ_ROPE if rope else 0, s))
        return k_dst, v_dst

    def validate(self, page_table, token_seq, token_pos, *, dst_page_table=None, stream=None):
        """(status, first bad token, code): code 1 sequence, 2 position, 3 source page, 4 destination page."""
        torch = _torch()
        n, batch, pt, ts, tp, dpt = self._tables(page_table, token_seq, token_pos, dst_page_table)
        bad, code = _i32(0), _i32(0)
        st = self._lib.kvshot_kv_project_validate(
            self._h, n, batch, pt, ts, tp, dpt, ctypes.byref(bad), ctypes.byref(code),
            stream if stream is not None else torch.cuda.current_stream().cuda_stream)
        if st not in (KVSHOT_OK, 5):
            _check("kvshot_kv_project_validate", st)
        return st, bad.value, code.value

    def set_option(self, option: int, value: int):
        _check("kvshot_kvproj_set_option", self._lib.kvshot_kvproj_set_option(self._h, option, value))

    def plan(self, n_tokens: int):
        s, p, t, w = _i32(0), _i32(0), _i32(0), _i32(0)
        _check("kvshot_kvproj_plan", self._lib.kvshot_kvproj_plan(self._h, n_tokens, ctypes.byref(s), ctypes.byref(p),
                                                                  ctypes.byref(t), ctypes.byref(w)))
        return dict(splits=s.value, path=p.value, tile_tokens=t.value, workgroups=w.value)

    def profile_read(self):
        a, c, k = ctypes.c_double(0), ctypes.c_double(0), _i64(0)
        _check("kvshot_kvproj_profile_read", self._lib.kvshot_kvproj_profile_read(
            self._h, ctypes.byref(a), ctypes.byref(c), ctypes.byref(k)))
        return dict(main_ms=a.value, combine_ms=c.value, calls=k.value)
