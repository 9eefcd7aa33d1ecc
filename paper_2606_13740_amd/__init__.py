"""Python binding of libdllm, the gfx950 denoising-step library.

Argument marshalling only: every function below forwards to the C ABI entry
point of the same name (see include/dllm.h) and every step runs in the HIP
kernels of ``csrc/``.  PyTorch supplies device memory and the stream.  There is
no fallback: if ``libdllm.so`` has not been built, importing the library fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdllm.so")

DLLM_OK, DLLM_E_INVAL, DLLM_E_CAPACITY, DLLM_E_DTYPE, DLLM_E_HIP, DLLM_E_UNIMPL, DLLM_E_NOMEM = 0, -1, -2, -3, -4, -5, -6
DLLM_F32, DLLM_BF16, DLLM_W8, DLLM_Q4 = 0, 1, 2, 3
K_QKV, K_ATTN, K_OPROJ, K_GATEUP, K_DOWN, K_LMHEAD = range(6)
KERNEL_CLASSES = {"qkv": K_QKV, "attn": K_ATTN, "oproj": K_OPROJ, "gateup": K_GATEUP, "down": K_DOWN,
                  "lmhead": K_LMHEAD}


class DllmError(RuntimeError):
    def __init__(self, code: int, func: str, msg: str):
        super().__init__(f"{func} failed with {code}: {msg}")
        self.code = code


class dllm_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("mask_id", ctypes.c_int32), ("block", ctypes.c_int32), ("eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("dtype", ctypes.c_int32), ("max_window", ctypes.c_int32),
                ("max_pos", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("qkv_bias", ctypes.c_int32)]


class dllm_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "ffn_norm",
                                               "bq", "bk", "bv")]


class dllm_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("layers", ctypes.POINTER(dllm_layer_weights))]


_lib = None
_vp, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t

_SIGNATURES = {
    "dllm_last_error": ([], ctypes.c_char_p),
    "dllm_version": ([], ctypes.c_char_p),
    "dllm_model_create": ([ctypes.POINTER(dllm_config), ctypes.POINTER(dllm_weights), _vp, ctypes.POINTER(_vp)],
                          ctypes.c_int),
    "dllm_model_destroy": ([_vp], ctypes.c_int),
    "dllm_kv_bytes": ([_vp, _i32, ctypes.POINTER(_sz)], ctypes.c_int),
    "dllm_kv_create": ([_vp, _vp, _sz, _i32, ctypes.POINTER(_vp)], ctypes.c_int),
    "dllm_kv_destroy": ([_vp], ctypes.c_int),
    "dllm_kv_prefix_len": ([_vp, ctypes.POINTER(_i32), ctypes.POINTER(_i32)], ctypes.c_int),
    "dllm_kv_set_prefix_len": ([_vp, _i32], ctypes.c_int),
    "dllm_prefill": ([_vp, _vp, _vp, _i32, _vp], ctypes.c_int),
    "dllm_denoise_step": ([_vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_commit": ([_vp, _vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_append_prefix_kv": ([_vp, _vp, _vp, _i32, _vp], ctypes.c_int),
    "dllm_refresh_kv": ([_vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_denoise_step_noalloc": ([_vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_denoise_window": ([_vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_denoise_window_sls": ([_vp, _vp, _i32, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_accept_drafts": ([_vp, _vp, _vp, _vp, _vp, _i32, ctypes.c_float, _vp, _vp, _vp], ctypes.c_int),
    "dllm_record_drafts": ([_vp, _vp, _vp, _i32, _vp], ctypes.c_int),
    "dllm_step_merged": ([_vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp],
                         ctypes.c_int),
    "dllm_debug_logits": ([_vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp], ctypes.c_int),
    "dllm_debug_hidden": ([_vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp], ctypes.c_int),
    "dllm_probe_enable": ([_vp, _i32, _i32], ctypes.c_int),
    "dllm_probe_read": ([_vp, ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "dllm_kernel_bytes": ([_vp, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "dllm_kernel_replay": ([_vp, _vp, _i32, _i32, _i32, _vp], ctypes.c_int),
    "dllm_read_bandwidth": ([_vp, ctypes.c_size_t, _vp, _vp], ctypes.c_int),
    "dllm_quantize_q4_0": ([_vp, _i32, _i32, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_quantize_int8": ([_vp, _i32, _i32, _i32, _vp, _vp, _vp], ctypes.c_int),
    "dllm_commit_staged": ([_vp, _vp, _vp, _vp, _vp, _i32, _i32, ctypes.c_float, ctypes.c_float, _vp, _vp, _vp],
                           ctypes.c_int),
}


def lib():
    """The loaded libdllm.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGNATURES.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(rc: int, func: str):
    if rc != DLLM_OK:
        raise DllmError(rc, func, lib().dllm_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


# ----------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ----------------------------------------------------------------------------


def dllm_model_create(cfg: dllm_config, weights: dllm_weights, stream=None) -> int:
    h = _vp()
    _check(lib().dllm_model_create(ctypes.byref(cfg), ctypes.byref(weights), _stream(stream), ctypes.byref(h)),
           "dllm_model_create")
    return h.value


def dllm_model_destroy(model: int):
    _check(lib().dllm_model_destroy(model), "dllm_model_destroy")


def dllm_kv_bytes(model: int, capacity: int) -> int:
    n = _sz()
    _check(lib().dllm_kv_bytes(model, capacity, ctypes.byref(n)), "dllm_kv_bytes")
    return n.value


def dllm_kv_create(model: int, buf, nbytes: int, capacity: int) -> int:
    h = _vp()
    _check(lib().dllm_kv_create(model, _ptr(buf), nbytes, capacity, ctypes.byref(h)), "dllm_kv_create")
    return h.value


def dllm_kv_destroy(kv: int):
    _check(lib().dllm_kv_destroy(kv), "dllm_kv_destroy")


def dllm_kv_prefix_len(kv: int):
    p, q = _i32(), _i32()
    _check(lib().dllm_kv_prefix_len(kv, ctypes.byref(p), ctypes.byref(q)), "dllm_kv_prefix_len")
    return p.value, q.value


def dllm_kv_set_prefix_len(kv: int, n: int):
    _check(lib().dllm_kv_set_prefix_len(kv, n), "dllm_kv_set_prefix_len")


def dllm_prefill(model: int, kv: int, ids, n: int, stream=None):
    _check(lib().dllm_prefill(model, kv, _ptr(ids), n, _stream(stream)), "dllm_prefill")


def dllm_denoise_step(model: int, kv: int, tok, mask, W: int, out_id, out_conf, stream=None):
    _check(lib().dllm_denoise_step(model, kv, _ptr(tok), _ptr(mask), W, _ptr(out_id), _ptr(out_conf),
                                   _stream(stream)), "dllm_denoise_step")


def dllm_denoise_step_noalloc(model: int, kv: int, tok, mask, W: int, out_id, out_conf, stream=None):
    _check(lib().dllm_denoise_step_noalloc(model, kv, _ptr(tok), _ptr(mask), W, _ptr(out_id), _ptr(out_conf),
                                           _stream(stream)), "dllm_denoise_step_noalloc")


def dllm_commit(conf, ids, tok, mask, seg_begin: int, seg_len: int, k: int, committed_pos=None,
                n_committed=None, stream=None):
    _check(lib().dllm_commit(_ptr(conf), _ptr(ids), _ptr(tok), _ptr(mask), seg_begin, seg_len, k,
                             _ptr(committed_pos), _ptr(n_committed), _stream(stream)), "dllm_commit")


def dllm_append_prefix_kv(model: int, kv: int, block_tok, n: int, stream=None):
    _check(lib().dllm_append_prefix_kv(model, kv, _ptr(block_tok), n, _stream(stream)), "dllm_append_prefix_kv")


def dllm_refresh_kv(model: int, kv: int, pos, new_ids, n: int, out_id=None, out_conf=None, stream=None):
    _check(lib().dllm_refresh_kv(model, kv, _ptr(pos), _ptr(new_ids), n, _ptr(out_id), _ptr(out_conf),
                                 _stream(stream)), "dllm_refresh_kv")


def dllm_denoise_window(model: int, kv: int, w0: int, tok, mask, W: int, out_id, out_conf, stream=None):
    _check(lib().dllm_denoise_window(model, kv, w0, _ptr(tok), _ptr(mask), W, _ptr(out_id), _ptr(out_conf),
                                     _stream(stream)), "dllm_denoise_window")


def dllm_denoise_window_sls(model: int, kv: int, w0: int, tok, mask, need, n_need: int, W: int, out_id, out_conf,
                            stream=None):
    _check(lib().dllm_denoise_window_sls(model, kv, w0, _ptr(tok), _ptr(mask), _ptr(need), n_need, W, _ptr(out_id),
                                         _ptr(out_conf), _stream(stream)), "dllm_denoise_window_sls")


def dllm_accept_drafts(conf, ids, draft_ids, tok, mask, n: int, theta: float, accepted_pos=None, n_accepted=None,
                       stream=None):
    _check(lib().dllm_accept_drafts(_ptr(conf), _ptr(ids), _ptr(draft_ids), _ptr(tok), _ptr(mask), n, float(theta),
                                    _ptr(accepted_pos), _ptr(n_accepted), _stream(stream)), "dllm_accept_drafts")


def dllm_record_drafts(ids, mask, draft_ids, n: int, stream=None):
    _check(lib().dllm_record_drafts(_ptr(ids), _ptr(mask), _ptr(draft_ids), n, _stream(stream)),
           "dllm_record_drafts")


def dllm_step_merged(model: int, kv: int, ref_pos, ref_ids, n_ref: int, block_tok, n_block: int, tok, mask,
                     W: int, out_id=None, out_conf=None, ref_out_id=None, ref_out_conf=None, stream=None):
    _check(lib().dllm_step_merged(model, kv, _ptr(ref_pos), _ptr(ref_ids), n_ref, _ptr(block_tok), n_block,
                                  _ptr(tok), _ptr(mask), W, _ptr(out_id), _ptr(out_conf), _ptr(ref_out_id),
                                  _ptr(ref_out_conf), _stream(stream)), "dllm_step_merged")


def dllm_debug_logits(model: int, kv: int, tok, mask, W: int, logits, out_id=None, out_conf=None, stream=None):
    _check(lib().dllm_debug_logits(model, kv, _ptr(tok), _ptr(mask), W, _ptr(logits), _ptr(out_id),
                                   _ptr(out_conf), _stream(stream)), "dllm_debug_logits")


def dllm_debug_hidden(model: int, kv: int, tok, mask, W: int, n_layers: int, x, stream=None):
    _check(lib().dllm_debug_hidden(model, kv, _ptr(tok), _ptr(mask), W, n_layers, _ptr(x), _stream(stream)),
           "dllm_debug_hidden")


def dllm_probe_enable(model: int, kernel_class: int, max_records: int):
    _check(lib().dllm_probe_enable(model, kernel_class, max_records), "dllm_probe_enable")


def dllm_probe_read(model: int):
    n, ms = _i32(), ctypes.c_double()
    _check(lib().dllm_probe_read(model, ctypes.byref(n), ctypes.byref(ms)), "dllm_probe_read")
    return n.value, ms.value


def dllm_kernel_replay(model: int, kv: int, kernel_class: int, W: int, n_launches: int, stream=None):
    _check(lib().dllm_kernel_replay(model, kv, kernel_class, W, n_launches, _stream(stream)), "dllm_kernel_replay")


def dllm_kernel_bytes(model: int, kernel_class: int, W: int, P: int) -> float:
    b = ctypes.c_double()
    _check(lib().dllm_kernel_bytes(model, kernel_class, W, P, ctypes.byref(b)), "dllm_kernel_bytes")
    return b.value


DLLM_TOKEN_INVISIBLE, DLLM_TOKEN_VISIBLE, DLLM_TOKEN_STABLE = 0, 1, 2


def dllm_commit_staged(conf, ids, tok, mask, state, seg_begin: int, seg_len: int, theta_visible: float,
                       theta_stable: float, promoted_pos=None, n_promoted=None, stream=None):
    _check(lib().dllm_commit_staged(_ptr(conf), _ptr(ids), _ptr(tok), _ptr(mask), _ptr(state), seg_begin, seg_len,
                                    theta_visible, theta_stable, _ptr(promoted_pos), _ptr(n_promoted),
                                    _stream(stream)), "dllm_commit_staged")


def dllm_quantize_q4_0(src, src_dtype: int, rows: int, K: int, codes, scales, stream=None):
    _check(lib().dllm_quantize_q4_0(_ptr(src), src_dtype, rows, K, _ptr(codes), _ptr(scales), _stream(stream)),
           "dllm_quantize_q4_0")


def dllm_quantize_int8(src, src_dtype: int, rows: int, K: int, codes, scales, stream=None):
    _check(lib().dllm_quantize_int8(_ptr(src), src_dtype, rows, K, _ptr(codes), _ptr(scales), _stream(stream)),
           "dllm_quantize_int8")


def dllm_read_bandwidth(buf, nbytes: int, sink, stream=None):
    _check(lib().dllm_read_bandwidth(_ptr(buf), nbytes, _ptr(sink), _stream(stream)), "dllm_read_bandwidth")


# ----------------------------------------------------------------------------
# Convenience holders: device weights and handles
# ----------------------------------------------------------------------------


DTYPES = {"f32": DLLM_F32, "bf16": DLLM_BF16, "w8": DLLM_W8, "q4": DLLM_Q4}


def make_config(shape, dtype: str, max_window: int = 64, max_pos: int = 8192) -> dllm_config:
    return dllm_config(shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ff, shape.vocab,
                       shape.mask_id, shape.block, shape.eps, shape.rope_base, DTYPES[dtype], max_window, max_pos,
                       getattr(shape, "n_kv_heads", 0), int(getattr(shape, "qkv_bias", False)))


class Model:
    """A library model built from host weight arrays (float32 or bf16 bit patterns).

    `layer_source(l)` may stream one layer at a time (dict of arrays) so that the
    device copy of the caller-side weights never exceeds one layer.
    """

    def __init__(self, shape, dtype: str, globals_: dict, layer_source, max_window: int = 64,
                 max_pos: int = 8192, device: str = "cuda"):
        import numpy as np
        import torch

        self.shape, self.dtype = shape, dtype
        self.cfg = make_config(shape, dtype, max_window, max_pos)
        dev = torch.device(device)

        def up(a):
            a = np.ascontiguousarray(a)
            if a.dtype == np.uint16:
                return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
            return torch.from_numpy(a.astype(np.float32, copy=False)).to(dev)

        keep = []
        LW = dllm_layer_weights * shape.n_layers
        layers = LW()
        # Weights are uploaded in full before create; large models pass them layer by layer
        # through the same create call by uploading everything first (device memory is ample).
        for l in range(shape.n_layers):
            src = layer_source(l)
            t = {k: up(v) for k, v in src.items()}
            keep.append(t)
            layers[l] = dllm_layer_weights(*[t[k].data_ptr() if k in t else None
                                             for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm",
                                                       "ffn_norm", "bq", "bk", "bv")])
        g = {k: up(v) for k, v in globals_.items()}
        keep.append(g)
        w = dllm_weights(g["embed"].data_ptr(), g["lm_head"].data_ptr(), g["final_norm"].data_ptr(), layers)
        stream = torch.cuda.current_stream()
        self.handle = dllm_model_create(self.cfg, w, stream)
        del keep
        torch.cuda.empty_cache()

    def close(self):
        if getattr(self, "handle", None):
            dllm_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KVCache:
    """A torch-allocated KV cache buffer wrapped by the library."""

    def __init__(self, model: Model, capacity: int, device: str = "cuda"):
        import torch

        self.model = model
        self.capacity = capacity
        self.nbytes = dllm_kv_bytes(model.handle, capacity)
        self.buf = torch.zeros(self.nbytes // 2 + 8, dtype=torch.int16, device=device)
        self.handle = dllm_kv_create(model.handle, self.buf, self.nbytes, capacity)

    @property
    def row_stride(self) -> int:
        return (self.capacity + 31) // 32 * 32

    def views(self):
        """(K [L][Hkv][Cs][Dh], V^T [L][Hkv][Dh][Cs]) as float32 tensors (Hkv K/V heads).

        fp32 models: views of the buffer.  bf16 / int8 / Q4_0 models: the fp16 planes,
        widened (a new tensor, not a view)."""
        import torch

        sh = self.model.shape
        Cs = self.row_stride
        Hkv = getattr(sh, "kv_heads", sh.n_heads)
        plane = Hkv * Cs * sh.head_dim
        if self.model.dtype == "f32":
            flat = self.buf.view(torch.uint8)[: sh.n_layers * 2 * plane * 4].view(torch.float32)
            per = flat.view(sh.n_layers, 2, plane)
            K, Vt = per[:, 0], per[:, 1]
        else:
            flat = self.buf.view(torch.uint8)[: sh.n_layers * 2 * plane * 2].view(torch.float16)
            per = flat.view(sh.n_layers, 2, plane).float()
            K, Vt = per[:, 0], per[:, 1]
        return (K.reshape(sh.n_layers, Hkv, Cs, sh.head_dim),
                Vt.reshape(sh.n_layers, Hkv, sh.head_dim, Cs))

    @property
    def prefix_len(self) -> int:
        return dllm_kv_prefix_len(self.handle)[0]

    @property
    def prompt_len(self) -> int:
        return dllm_kv_prefix_len(self.handle)[1]

    def close(self):
        if getattr(self, "handle", None):
            dllm_kv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
