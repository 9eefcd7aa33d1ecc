"""Seeded synthetic inputs shared by the oracle and the GPU path.

This module only *draws* inputs: model shapes, random weights, prompt ids,
block tokens with mask flags, and refresh picks.  It holds none of the
diffusion-LLM arithmetic (no norm, projection, attention, softmax or commit),
so the oracle and the HIP path may both import it without sharing any of the
method.

Weights are i.i.d. N(0, 0.02^2) draws from the counter-based generator in
``_gen.c`` (SplitMix64 + Box-Muller), one stream per tensor, so any tensor can
be regenerated on its own and in parallel.  bf16 models round each fp32 draw to
bfloat16 (round to nearest even).  Norm gains are ones.  Token ids are uniform.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, Iterable, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


def build_generator(verbose: bool = False) -> str:
    """Compile ``_gen.c`` into ``libsynth.so`` (gcc, OpenMP)."""
    import subprocess

    src = os.path.join(_HERE, "_gen.c")
    out = os.path.join(_HERE, "libsynth.so")
    cmd = ["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", src, "-o", out + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libsynth.so")
        if not os.path.exists(path):
            build_generator()
        lib = ctypes.CDLL(path)
        u64, f32, vp = ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p
        lib.synth_normal_f32.argtypes = [u64, u64, u64, u64, f32, vp]
        lib.synth_normal_bf16.argtypes = [u64, u64, u64, u64, f32, vp]
        lib.synth_uniform_int.argtypes = [u64, u64, u64, u64, u64, vp]
        lib.synth_set_threads.argtypes = [ctypes.c_int]
        threads = int(os.environ.get("SYNTH_THREADS", "0") or 0)
        if threads <= 0:
            threads = min(os.cpu_count() or 1, 16)
        lib.synth_set_threads(threads)
        _LIB = lib
    return _LIB


# ----------------------------------------------------------------------------
# Model shapes
# ----------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Shape:
    """Transformer shape of a LLaDA-style masked-diffusion LM."""

    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    mask_id: int
    eps: float = 1e-5
    rope_base: float = 10000.0
    block: int = 32
    n_kv_heads: int = 0          # K/V heads (grouped-query attention); 0 = n_heads
    qkv_bias: bool = False       # biases on the Q, K and V projections

    def __post_init__(self):
        assert self.n_heads * self.head_dim == self.d_model
        assert 0 <= self.mask_id < self.vocab
        assert self.kv_heads >= 1 and self.n_heads % self.kv_heads == 0

    def with_layers(self, n_layers: int) -> "Shape":
        return dataclasses.replace(self, n_layers=n_layers)

    @property
    def kv_heads(self) -> int:
        return self.n_kv_heads or self.n_heads

    @property
    def d_kv(self) -> int:
        return self.kv_heads * self.head_dim

    @property
    def params_per_layer(self) -> int:
        d, f = self.d_model, self.d_ff
        return 2 * d * d + 2 * d * self.d_kv + 3 * f * d


# Tiny fp32 model: 2 layers, d 256, 4 heads x 64, FFN 688, vocab 1024 (1023 = MASK).
TINY = Shape(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ff=688, vocab=1024, mask_id=1023)

# LLaDA-8B shape: 32 layers, d 4096, 32 heads x 128, FFN 12288, vocab 126464.
# The MASK id is taken as vocab - 1, mirroring the tiny model.
LLADA_8B = Shape(n_layers=32, d_model=4096, n_heads=32, head_dim=128, d_ff=12288, vocab=126464,
                 mask_id=126463)

# Small shapes for fast tests; they exercise ragged tiles (d_ff, vocab not tile multiples).
MICRO = Shape(n_layers=2, d_model=64, n_heads=2, head_dim=32, d_ff=96, vocab=80, mask_id=79)
SMALL_BF16 = Shape(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ff=688, vocab=1000, mask_id=999)

# Dream-7B shape (grouped-query attention): 28 layers, d 3584, 28 query heads x 128
# sharing 4 K/V heads, FFN 18944, vocab 152064, RoPE base 1e6, RMSNorm eps 1e-6,
# biases on Q/K/V.  MASK = vocab - 1 as for the other shapes.
DREAM_7B = Shape(n_layers=28, d_model=3584, n_heads=28, head_dim=128, d_ff=18944, vocab=152064, mask_id=152063,
                 eps=1e-6, rope_base=1e6, n_kv_heads=4, qkv_bias=True)

# Small grouped-query shapes: 2 query heads per K/V head (fp32 and bf16), and one
# K/V head for 4 query heads (multi-query) with ragged FFN and vocab tiles.
TINY_GQA = Shape(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ff=688, vocab=1024, mask_id=1023,
                 n_kv_heads=2, qkv_bias=True)
SMALL_MQA = Shape(n_layers=2, d_model=512, n_heads=4, head_dim=128, d_ff=688, vocab=1000, mask_id=999,
                  n_kv_heads=1, qkv_bias=True)
MICRO_GQA = Shape(n_layers=2, d_model=64, n_heads=4, head_dim=16, d_ff=96, vocab=80, mask_id=79, n_kv_heads=2,
                  qkv_bias=True)

PRESETS = {"tiny": TINY, "llada8b": LLADA_8B, "micro": MICRO, "small": SMALL_BF16, "dream7b": DREAM_7B,
           "tiny_gqa": TINY_GQA, "small_mqa": SMALL_MQA}

WEIGHT_STD = 0.02

# Per-layer tensors in a fixed order; the index feeds the stream id.
LAYER_TENSORS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
LAYER_BIASES = ("bq", "bk", "bv")       # fp32 draws, present when shape.qkv_bias
LAYER_GAINS = ("attn_norm", "ffn_norm")


def tensor_shape(shape: Shape, name: str):
    d, f, v, dkv = shape.d_model, shape.d_ff, shape.vocab, shape.d_kv
    return {
        "embed": (v, d), "lm_head": (v, d), "final_norm": (d,),
        "wq": (d, d), "wk": (dkv, d), "wv": (dkv, d), "wo": (d, d),
        "wg": (f, d), "wu": (f, d), "wd": (d, f),
        "bq": (d,), "bk": (dkv,), "bv": (dkv,),
        "attn_norm": (d,), "ffn_norm": (d,),
    }[name]


def _stream_id(name: str, layer: int) -> int:
    if name == "embed":
        return 1
    if name == "lm_head":
        return 2
    return 1000 + 16 * layer + (LAYER_TENSORS + LAYER_BIASES).index(name)


def normal(seed: int, stream: int, n: int, dtype: str, offset: int = 0,
           std: float = WEIGHT_STD, out: Optional[np.ndarray] = None) -> np.ndarray:
    """n draws of N(0, std^2); dtype 'f32' -> float32, 'bf16' -> uint16 bit patterns."""
    lib = _lib()
    if dtype == "f32":
        arr = out if out is not None else np.empty(n, np.float32)
        assert arr.dtype == np.float32 and arr.size == n and arr.flags.c_contiguous
        lib.synth_normal_f32(seed, stream, offset, n, std, arr.ctypes.data)
    elif dtype == "bf16":
        arr = out if out is not None else np.empty(n, np.uint16)
        assert arr.dtype == np.uint16 and arr.size == n and arr.flags.c_contiguous
        lib.synth_normal_bf16(seed, stream, offset, n, std, arr.ctypes.data)
    else:
        raise ValueError(dtype)
    return arr


def weight(shape: Shape, name: str, layer: int = -1, dtype: str = "f32", seed: int = 0,
           out: Optional[np.ndarray] = None) -> np.ndarray:
    """One weight tensor (row-major [out][in]); gains are ones."""
    shp = tensor_shape(shape, name)
    if name in LAYER_GAINS or name == "final_norm":
        return np.ones(shp, np.float32)
    n = int(np.prod(shp))
    return normal(seed, _stream_id(name, layer), n, dtype, out=out).reshape(shp)


def layer_weights(shape: Shape, layer: int, dtype: str = "f32", seed: int = 0) -> Dict[str, np.ndarray]:
    w = {n: weight(shape, n, layer, dtype, seed) for n in LAYER_TENSORS}
    if shape.qkv_bias:
        for b in LAYER_BIASES:
            w[b] = weight(shape, b, layer, "f32", seed)
    for g in LAYER_GAINS:
        w[g] = weight(shape, g, layer)
    return w


def global_weights(shape: Shape, dtype: str = "f32", seed: int = 0) -> Dict[str, np.ndarray]:
    return {
        "embed": weight(shape, "embed", -1, dtype, seed),
        "lm_head": weight(shape, "lm_head", -1, dtype, seed),
        "final_norm": weight(shape, "final_norm"),
    }


def all_weights(shape: Shape, dtype: str = "f32", seed: int = 0) -> dict:
    """{'embed','lm_head','final_norm','layers': [per-layer dicts]}."""
    w = global_weights(shape, dtype, seed)
    w["layers"] = [layer_weights(shape, l, dtype, seed) for l in range(shape.n_layers)]
    return w


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float32."""
    return (np.ascontiguousarray(u).astype(np.uint32) << 16).view(np.float32)


def as_f32(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(a) if a.dtype == np.uint16 else a.astype(np.float32, copy=False)


# ----------------------------------------------------------------------------
# Token inputs
# ----------------------------------------------------------------------------


def uniform_ids(seed: int, stream: int, n: int, hi: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, np.int32)
    if n:
        _lib().synth_uniform_int(seed, stream, offset, n, hi, out.ctypes.data)
    return out


PROMPT_SEED, BLOCK_SEED, REFRESH_SEED = 1, 2, 3


def prompt_ids(shape: Shape, n: int, seed: int = PROMPT_SEED) -> np.ndarray:
    """n prompt ids, uniform over the non-MASK ids [0, mask_id)."""
    return uniform_ids(seed, 10, n, shape.mask_id)


def window(shape: Shape, n_rows: int, masked: Iterable[int], seed: int = BLOCK_SEED):
    """(tok int32[n], mask uint8[n]): random committed ids, MASK at `masked`."""
    tok = uniform_ids(seed, 20, n_rows, shape.mask_id)
    mask = np.zeros(n_rows, np.uint8)
    for i in masked:
        mask[i] = 1
        tok[i] = shape.mask_id
    return tok, mask


def refresh_picks(shape: Shape, block_begin: int, block_len: int, n: int, call: int,
                  seed: int = REFRESH_SEED):
    """n distinct positions in [block_begin, block_begin+block_len) and new ids."""
    r = uniform_ids(seed, 30 + 2 * call, 4 * block_len, 1 << 30)
    order = np.argsort(r[:block_len], kind="stable")
    pos = (block_begin + order[:n]).astype(np.int32)
    new_ids = uniform_ids(seed, 31 + 2 * call, n, shape.mask_id)
    return pos, new_ids
