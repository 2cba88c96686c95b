"""C ABI checks that need no GPU: the library loads, exports every declared
function, and rejects bad arguments on the host before touching a device."""
import ctypes
import os
import re

import pytest

import paper_2604_26412_amd as K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(K.LIB_PATH):
        from paper_2604_26412_amd import build
        build.build()
    return K.load_library()


def declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z_0-9]*\s*\*?\s*(kvshot_[a-z_0-9]+)\s*\(", text,
                                flags=re.M)
    return sorted(set(names))


def test_header_declares_the_binding_symbols():
    assert declared_functions() == sorted(K.EXPORTED_SYMBOLS)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def good_cfg(**kw):
    c = K.KvshotConfig()
    c.num_q_heads, c.num_kv_heads, c.head_dim, c.page_size = 32, 8, 128, 16
    c.dtype, c.out_dtype, c.max_batch, c.max_draft = 0, 0, 4, 8
    c.max_pages_per_seq, c.num_pages, c.max_position = 16, 64, 300
    c.rope_theta, c.softmax_scale, c.reserved = 1e6, 0.0, 0
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), 2),
    (dict(num_q_heads=30), 1),
    (dict(num_q_heads=128, num_kv_heads=8), 2),
    (dict(page_size=24), 1),
    (dict(page_size=8), 1),
    (dict(page_size=512), 1),
    (dict(max_draft=65), 1),
    (dict(max_draft=0), 1),
    (dict(dtype=7), 1),
    (dict(out_dtype=-1), 1),
    (dict(max_batch=0), 1),
    (dict(num_pages=0), 1),
    (dict(max_position=0), 1),
    (dict(rope_theta=0.0), 1),
    (dict(rope_theta=float("nan")), 1),
    (dict(softmax_scale=-1.0), 1),
    (dict(reserved=3), 1),
    (dict(slot_stride=100), 1),
])
def test_init_rejects_bad_configs_before_any_device_call(lib, kw, status):
    h = ctypes.c_void_p(123)
    assert lib.kvshot_draft_attn_init(ctypes.byref(good_cfg(**kw)), ctypes.byref(h)) == status
    assert h.value is None


def test_null_arguments(lib):
    h = ctypes.c_void_p()
    assert lib.kvshot_draft_attn_init(None, ctypes.byref(h)) == 1
    assert lib.kvshot_draft_attn_init(ctypes.byref(good_cfg()), None) == 1
    assert lib.kvshot_draft_attn_step(None, 1, 1, 16, *([None] * 10), None) == 1
    assert lib.kvshot_draft_attn_tree(None, 1, 1, 16, *([None] * 10), None) == 1
    assert lib.kvshot_draft_attn_set_option(None, 0, 0) == 1
    assert lib.kvshot_draft_attn_plan(None, 1, 1, 16, None, None, None, None) == 1
    assert lib.kvshot_draft_attn_profile_read(None, None, None, None) == 1
    assert lib.kvshot_debug_tree_mask(None, 1, 1, None, None, None, None) == 1
    assert lib.kvshot_debug_gather_kv(None, 1, 1, *([None] * 7)) == 1
    assert lib.kvshot_debug_mfma_rate(0, 1, None, None) == 1
    assert lib.kvshot_debug_mfma_rate(1, 0, None, None) == 1
    assert lib.kvshot_draft_attn_validate(None, 1, 1, 16, None, None, None, None, None, None) == 1
    assert lib.kvshot_draft_attn_destroy(None) == 0


def test_status_strings(lib):
    assert lib.kvshot_status_string(0) == b"ok"
    assert lib.kvshot_status_string(5).startswith(b"contract")
    assert lib.kvshot_status_string(99) == b"unknown status"


def test_config_struct_layout_matches_header():
    # int32 x10, int64, double, float, int32, int64 x3
    assert ctypes.sizeof(K.KvshotConfig) == 10 * 4 + 8 + 8 + 4 + 4 + 3 * 8
    assert K.KvshotConfig.max_position.offset == 40
    assert K.KvshotConfig.page_stride.offset == 64


def test_product_path_does_not_import_the_oracle():
    src = open(os.path.join(ROOT, "paper_2604_26412_amd", "__init__.py")).read()
    assert "oracle" not in src.replace("no fallback", "")
    for fn in os.listdir(os.path.join(ROOT, "paper_2604_26412_amd", "csrc")):
        assert "oracle" not in open(os.path.join(ROOT, "paper_2604_26412_amd", "csrc", fn)).read().lower()


def test_binding_argument_counts_match_header(lib):
    text = ""
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text += open(os.path.join(ROOT, "include", fn)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    for name in declared_functions():
        m = re.search(name + r"\s*\(([^;]*?)\)\s*;", text, flags=re.S)
        assert m, name
        params = [p for p in m.group(1).split(",") if p.strip() and p.strip() != "void"]
        assert len(getattr(lib, name).argtypes) == len(params), name


@pytest.mark.parametrize("d,max_tokens", [(0, 8), (100, 8), (384, 8), (256, 0), (-256, 8)])
def test_fusion_init_rejects_bad_sizes_before_any_device_call(lib, d, max_tokens):
    h = ctypes.c_void_p(123)
    assert lib.kvshot_fusion_init(d, max_tokens, ctypes.byref(h)) == 1
    assert h.value is None


def test_fusion_null_handle(lib):
    assert lib.kvshot_gated_delta_fusion(None, 1, None, None, None, None, None, None, None, 0, None) == 1
    assert lib.kvshot_fusion_set_option(None, 0, 0) == 1
    assert lib.kvshot_fusion_plan(None, 1, None, None) == 1
    assert lib.kvshot_fusion_destroy(None) == 0


def test_call_struct_layout_matches_the_header():
    # six int32 fields, then thirteen pointers: 24 + 13 * 8 bytes, pointers 8-aligned
    assert ctypes.sizeof(K.KvshotCall) == 128
    assert K.KvshotCall.q.offset == 24 and K.KvshotCall.lse.offset == 120
    text = open(os.path.join(ROOT, "include", "kvshot_draft_attn.h")).read()
    body = text[text.index("typedef struct kvshot_call {"):text.index("} kvshot_call;")]
    fields = re.findall(r"^\s*(?:const\s+)?[a-z0-9_]+\s*\*?\s*([a-z_0-9]+);", body, flags=re.M)
    assert fields == [f for f, _ in K.KvshotCall._fields_]


def test_call_rejects_null_struct_and_handle(lib):
    assert lib.kvshot_draft_attn_call(None, None, None) == 1
    assert lib.kvshot_draft_attn_validate_call(None, None, None, None) == 1


def good_proj_cfg(**kw):
    c = K.KvprojConfig()
    c.num_kv_heads, c.head_dim, c.num_layers, c.page_size = 8, 128, 3, 16
    c.max_pages_per_seq, c.num_pages, c.dst_num_pages, c.max_tokens = 16, 64, 64, 512
    c.max_position, c.rope_theta = 300, 1e6
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=64), 2),
    (dict(num_kv_heads=0), 1),
    (dict(num_kv_heads=17), 1),
    (dict(num_layers=0), 1),
    (dict(num_layers=5), 1),
    (dict(page_size=24), 1),
    (dict(page_size=8), 1),
    (dict(num_pages=0), 1),
    (dict(dst_num_pages=0), 1),
    (dict(max_tokens=0), 1),
    (dict(max_position=0), 1),
    (dict(rope_theta=-1.0), 1),
    (dict(slot_stride=64), 1),
    (dict(dst_head_stride=12), 1),
])
def test_kvproj_init_rejects_bad_configs_before_any_device_call(lib, kw, status):
    h = ctypes.c_void_p(123)
    assert lib.kvshot_kvproj_init(ctypes.byref(good_proj_cfg(**kw)), ctypes.byref(h)) == status
    assert h.value is None


def test_kvproj_null_handle(lib):
    h = ctypes.c_void_p()
    assert lib.kvshot_kvproj_init(None, ctypes.byref(h)) == 1
    assert lib.kvshot_kv_project(None, 1, 1, None, None, *([None] * 8), 0, None) == 1
    assert lib.kvshot_kv_project_validate(None, 1, 1, None, None, None, None, None, None, None) == 1
    assert lib.kvshot_kvproj_set_option(None, 0, 0) == 1
    assert lib.kvshot_kvproj_plan(None, 1, None, None, None, None) == 1
    assert lib.kvshot_kvproj_profile_read(None, None, None, None) == 1
    assert lib.kvshot_kvproj_destroy(None) == 0


def test_kvproj_config_struct_layout_matches_the_header():
    # int32 x8, int64, double, int64 x6
    assert ctypes.sizeof(K.KvprojConfig) == 8 * 4 + 8 + 8 + 6 * 8
    text = open(os.path.join(ROOT, "include", "kvshot_kvproj.h")).read()
    body = text[text.index("typedef struct kvshot_kvproj_config {"):text.index("} kvshot_kvproj_config;")]
    fields = re.findall(r"^\s*[a-z0-9_]+\s+([a-z_0-9]+);", body, flags=re.M)
    assert fields == [f for f, _ in K.KvprojConfig._fields_]


def test_acceptance_stats_rejects_bad_arguments_before_any_device_call(lib):
    f = lib.kvshot_acceptance_stats
    ok = ctypes.c_void_p(64)    # aligned, never dereferenced: every case below fails on the host
    assert f(None, -1, 7, ok, ok, ok, None, 0, None) == 1
    assert f(None, 5, 7, ok, ok, ok, None, 0, None) == 1          # records missing
    assert f(ok, 5, 0, ok, ok, ok, None, 0, None) == 1            # K out of range
    assert f(ok, 5, 256, ok, ok, ok, None, 0, None) == 1
    assert f(ok, 5, 7, None, ok, ok, None, 0, None) == 1
    assert f(ok, 5, 7, ok, ok, ok, ok, 7, None) == 1              # retention step past K - 1
    assert f(ctypes.c_void_p(66), 5, 7, ok, ok, ok, None, 0, None) == 1   # misaligned


def test_topk_workspace_sizes(lib):
    f = lib.kvshot_topk_workspace_bytes
    assert f(80, 16384) == 0                       # one chunk: finished in place
    assert f(80, 16385) == 80 * 2 * 136
    assert f(80, 151936) == 80 * 10 * 136
    assert f(1, 64 * 16384) == 64 * 136
    assert f(1, 64 * 16384 + 1) == -1 and f(0, 100) == -1 and f(3, 0) == -1


def test_tree_calls_reject_bad_arguments_before_any_device_call(lib):
    ok = ctypes.c_void_p(256)   # aligned, never dereferenced: every case below fails on the host
    top = lib.kvshot_topk_logprobs
    assert top(ok, 0, 4, 100, 104, 17, ok, ok, None, 0, None) == 1        # k > 16
    assert top(ok, 0, 4, 100, 104, 0, ok, ok, None, 0, None) == 1
    assert top(ok, 0, 4, 5, 8, 6, ok, ok, None, 0, None) == 1             # k > vocab
    assert top(ok, 1, 4, 100, 99, 4, ok, ok, None, 0, None) == 1          # stride < vocab
    assert top(ctypes.c_void_p(257), 0, 4, 100, 104, 4, ok, ok, None, 0, None) == 1   # bf16 not 2-byte aligned
    assert top(ctypes.c_void_p(258), 1, 4, 100, 104, 4, ok, ok, None, 0, None) == 1   # float32 not 4-byte aligned
    assert top(ok, 7, 4, 100, 104, 4, ok, ok, None, 0, None) == 1         # dtype
    assert top(ok, 0, 4, 20000, 20000, 4, ok, ok, None, 0, None) == 1     # workspace missing
    need = lib.kvshot_topk_workspace_bytes(4, 20000)
    assert top(ok, 0, 4, 20000, 20000, 4, ok, ok, ok, need - 1, None) == 1
    assert top(None, 0, 4, 100, 104, 4, ok, ok, None, 0, None) == 1
    ex = lib.kvshot_tree_expand
    assert ex(2, 17, 10, 10, ok, ok, ok, ok, ok, ok, None) == 1           # frontier > 16
    assert ex(2, 10, 17, 10, ok, ok, ok, ok, ok, ok, None) == 1
    assert ex(2, 1, 4, 5, ok, ok, ok, ok, ok, ok, None) == 1              # k > frontier * proposals
    assert ex(2, 10, 10, 17, ok, ok, ok, ok, ok, ok, None) == 1
    assert ex(0, 10, 10, 10, ok, ok, ok, ok, ok, ok, None) == 1
    assert ex(2, 10, 10, 10, ok, ok, None, ok, ok, ok, None) == 1
    sel = lib.kvshot_tree_select
    assert sel(2, 17, 16, 60, ok, ok, ok, ok, ok, ok, ok, None) == 1      # depth * k > 256
    assert sel(2, 8, 10, 81, ok, ok, ok, ok, ok, ok, ok, None) == 1       # n > depth * k
    assert sel(2, 8, 10, 0, ok, ok, ok, ok, ok, ok, ok, None) == 1
    assert sel(2, 8, 10, 60, ok, ok, ok, ok, ok, None, ok, None) == 1


def test_tree_level_workspace_sizes_and_rejections(lib):
    f = lib.kvshot_tree_level_workspace_bytes
    assert f(8, 10, 151936) == 8 * 17 * 256 + 8 * 10 * 11 * 136
    assert f(65, 1, 100) == 65 * 17 * 256 + 65 * 2 * 136
    assert f(0, 10, 100) == -1 and f(8, 17, 100) == -1 and f(8, 10, 64 * 16384 + 1) == -1
    ok = ctypes.c_void_p(256)
    lv = lib.kvshot_tree_level
    need = f(2, 10, 100)
    assert lv(ok, 0, 2, 17, 100, 104, 10, ok, ok, ok, ok, ok, need, None) == 1          # frontier > 16
    assert lv(ok, 0, 2, 10, 100, 104, 17, ok, ok, ok, ok, ok, need, None) == 1          # k > 16
    assert lv(ok, 0, 2, 10, 5, 8, 10, ok, ok, ok, ok, ok, need, None) == 1              # k > vocab
    assert lv(ok, 0, 2, 10, 100, 104, 10, ok, ok, ok, ok, ok, need - 1, None) == 1      # workspace too small
    assert lv(ok, 0, 2, 10, 100, 104, 10, ok, ok, ok, ok, ctypes.c_void_p(264), need, None) == 1   # not 256-aligned
    assert lv(ok, 0, 2, 10, 100, 104, 10, None, ok, ok, ok, ok, need, None) == 1        # scores missing
    assert lv(ok, 0, 0, 10, 100, 104, 10, ok, ok, ok, ok, ok, need, None) == 1
