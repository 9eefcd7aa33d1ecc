"""The C ABI without a GPU: the library loads, exports every function the header
declares, and rejects bad arguments on the host before any GPU work."""
import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dllm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dllm_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def dl():
    import paper_2606_13740_amd as pkg
    try:
        pkg.lib()
    except ImportError:
        pytest.skip("libdllm.so not built")
    return pkg


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("dllm_denoise_step", "dllm_commit", "dllm_append_prefix_kv", "dllm_refresh_kv",
                     "dllm_prefill", "dllm_model_create", "dllm_kv_create"):
        assert required in names


def test_library_exports_every_declared_symbol(dl):
    lib = ctypes.CDLL(dl.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_wraps_every_declared_symbol(dl):
    missing = [n for n in declared_functions() if n not in dl._SIGNATURES]
    assert not missing, missing


def _create(dl, cfg):
    h = ctypes.c_void_p()
    rc = dl.lib().dllm_model_create(ctypes.byref(cfg), None, None, ctypes.byref(h))
    return rc, dl.lib().dllm_last_error().decode()


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 48, -1),          # d_model != heads * head_dim
    ("mask_id", 1024, -1),         # outside the vocabulary
    ("max_window", 0, -1),
    ("max_window", 257, -1),
    ("dtype", 7, -3),
    ("eps", 0.0, -1),
    ("block", 0, -1),
    ("n_kv_heads", 3, -1),         # does not divide 4 query heads
    ("n_kv_heads", 8, -1),         # more K/V heads than query heads
    ("n_kv_heads", -1, -1),
    ("qkv_bias", 2, -1),
])
def test_model_create_validates_config(dl, field, value, code):
    cfg = dl.make_config(synth.TINY, "f32")
    setattr(cfg, field, value)
    rc, msg = _create(dl, cfg)
    assert rc == code and msg


def test_model_create_rejects_null_weights(dl):
    cfg = dl.make_config(synth.TINY, "f32")
    rc, msg = _create(dl, cfg)
    assert rc == dl.DLLM_E_INVAL and "weights" in msg


def test_bf16_head_dim_support_is_checked(dl):
    cfg = dl.make_config(synth.MICRO, "bf16")       # head_dim 32: fp32 only
    rc, _ = _create(dl, cfg)
    assert rc == dl.DLLM_E_DTYPE


@pytest.mark.parametrize("args,code", [
    ((1, 1, 1, 1, 0, 4, -1), -1),        # k < 0
    ((1, 1, 1, 1, -1, 4, 1), -1),        # seg_begin < 0
    ((1, 1, 1, 1, 0, 2000, 1), -1),      # segment too long
    ((None, 1, 1, 1, 0, 4, 1), -1),      # null pointer
])
def test_commit_validates_on_host(dl, args, code):
    rc = dl.lib().dllm_commit(*args, None, None, None)
    assert rc == code and dl.lib().dllm_last_error()


def test_null_handles_are_rejected(dl):
    L = dl.lib()
    n = ctypes.c_size_t()
    assert L.dllm_kv_bytes(None, 16, ctypes.byref(n)) == dl.DLLM_E_INVAL
    assert L.dllm_denoise_step(None, None, None, None, 32, None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_append_prefix_kv(None, None, None, 32, None) == dl.DLLM_E_INVAL
    assert L.dllm_refresh_kv(None, None, None, None, 4, None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_step_merged(None, None, None, None, 0, None, 32, None, None, 0, None, None, None, None,
                              None) == dl.DLLM_E_INVAL
    assert L.dllm_denoise_window(None, None, 0, None, None, 32, None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_denoise_window_sls(None, None, 0, None, None, None, 0, 32, None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_kernel_replay(None, None, 0, 32, 1, None) == dl.DLLM_E_INVAL


def test_draft_calls_validate_on_host(dl):
    L = dl.lib()
    buf = (ctypes.c_int32 * 8)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    assert L.dllm_accept_drafts(None, p, p, p, p, 4, ctypes.c_float(0.5), None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_accept_drafts(p, p, p, p, p, 0, ctypes.c_float(0.5), None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_accept_drafts(p, p, p, p, p, 1025, ctypes.c_float(0.5), None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_accept_drafts(p, p, p, p, p, 4, ctypes.c_float(float("nan")), None, None, None) == dl.DLLM_E_INVAL
    assert L.dllm_record_drafts(p, None, p, 4, None) == dl.DLLM_E_INVAL
    assert L.dllm_record_drafts(p, p, p, 0, None) == dl.DLLM_E_INVAL
    assert L.dllm_prefill(None, None, None, 4, None) == dl.DLLM_E_INVAL
    assert L.dllm_kv_set_prefix_len(None, 0) == dl.DLLM_E_INVAL
    assert L.dllm_model_destroy(None) == dl.DLLM_OK
    assert L.dllm_kv_destroy(None) == dl.DLLM_OK


def test_read_bandwidth_validates_on_host(dl):
    L = dl.lib()
    assert L.dllm_read_bandwidth(None, 16, None, None) == dl.DLLM_E_INVAL
    # misaligned buffer / size: rejected before any launch (the pointers are never dereferenced)
    assert L.dllm_read_bandwidth(ctypes.c_void_p(0x1001), 16, ctypes.c_void_p(0x2000), None) == dl.DLLM_E_INVAL
    assert L.dllm_read_bandwidth(ctypes.c_void_p(0x1000), 17, ctypes.c_void_p(0x2000), None) == dl.DLLM_E_INVAL


@pytest.mark.parametrize("args,code", [
    ((None, 1, 1, 1, 1, 0, 4, 0.7, 0.9), -1),          # null pointer
    ((1, 1, 1, 1, 1, 0, 0, 0.7, 0.9), -1),             # empty segment
    ((1, 1, 1, 1, 1, 0, 1025, 0.7, 0.9), -1),          # segment too long
    ((1, 1, 1, 1, 1, -1, 4, 0.7, 0.9), -1),            # negative begin
    ((1, 1, 1, 1, 1, 0, 4, float("nan"), 0.9), -1),    # non-finite threshold
])
def test_commit_staged_validates_on_host(dl, args, code):
    rc = dl.lib().dllm_commit_staged(*args, None, None, None)
    assert rc == code and dl.lib().dllm_last_error()


def test_version_string(dl):
    assert dl.lib().dllm_version().startswith(b"dllm")


def test_quantizers_validate_on_host(dl):
    L = dl.lib()
    p = ctypes.c_void_p(0x1000)
    for f in (L.dllm_quantize_int8, L.dllm_quantize_q4_0):
        assert f(None, dl.DLLM_BF16, 4, 4, p, p, None) == dl.DLLM_E_INVAL
        assert f(p, dl.DLLM_BF16, 0, 4, p, p, None) == dl.DLLM_E_INVAL
        assert f(p, dl.DLLM_BF16, 4, 0, p, p, None) == dl.DLLM_E_INVAL
        assert f(p, dl.DLLM_W8, 4, 4, p, p, None) == dl.DLLM_E_DTYPE
