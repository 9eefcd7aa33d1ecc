"""Oracle for the denoising step of block-wise diffusion-LLM inference.

TEST INFRASTRUCTURE.  This package is a plain, slow, float64 NumPy statement of
what the GPU path computes.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path never does, and it shares no
code with the HIP kernels or their runtime.  Its only shared dependency is the
seeded input generator (``synth``), which draws inputs and holds none of the
method.

What is computed (paper: Background, "Block-Wise Decoding"; System Design,
"Overview" and "Multi-Block Speculative Decoding"; Implementation):
  * the output is split into consecutive blocks decoded left to right; tokens
    of the current block are predicted in parallel at every denoising step and a
    confidence-selected subset of the masked ones is committed;
  * completed blocks are kept as a reused prefix KV cache, and one step runs the
    transformer only over the current decoding window, which attends to that
    prefix and globally (bidirectionally) within itself;
  * a window may hold speculative draft tokens of the next block; drafts never
    write the prefix cache;
  * revised positions have their confidence, identity and KV recomputed sparsely
    and the result is visible from the next step on (Dual-Path Progressive
    Revision, "Sparse Cache Refresh").

The paper gives no architecture beyond naming LLaDA-8B and its operators
(RMSNorm, matrix multiplication, FlashAttention); the model below is the
pre-norm LLaMA-style block those operators make up: RMSNorm, multi-head
attention with rotate-half RoPE, SwiGLU FFN, no biases, untied LM head.

Readings taken where the paper is silent:
  * confidence of a position = softmax probability of its argmax token at
    temperature 0, with the MASK id excluded from the softmax;
  * argmax ties go to the lowest id; commit ties go to the lower position;
  * prefix rows see keys block-causally (the prompt is one bidirectional block,
    block b sees every block <= b); the window sees every key in [0, P + W);
  * a refresh scatters the new K/V of every refreshed row at a layer before that
    layer's attention, and each refreshed row attends to the keys up to the end
    of its own block.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

NEG_INF = -np.inf


# -----------------------------------------------------------------------------
# Operators (Implementation section: RMSNorm, matmul, attention, elementwise)
# -----------------------------------------------------------------------------


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g, over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope(u: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of u[n, H, Dh] at absolute positions pos[n].

    For j < Dh/2 the pair (u_j, u_{j+Dh/2}) is rotated by theta = pos * base^(-2j/Dh).
    """
    dh = u.shape[-1]
    half = dh // 2
    j = np.arange(half, dtype=np.float64)
    theta = pos.astype(np.float64)[:, None] * base ** (-2.0 * j / dh)   # [n, half]
    c = np.cos(theta)[:, None, :]
    s = np.sin(theta)[:, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def softmax(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def group_heads(KV: np.ndarray, n_heads: int) -> np.ndarray:
    """Grouped-query attention: K or V [keys, Hkv, Dh] seen by n_heads query heads;
    query head h reads K/V head h // (n_heads / Hkv).  Hkv = n_heads is plain
    multi-head attention."""
    G = n_heads // KV.shape[1]
    return np.repeat(KV, G, axis=1)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, limits: np.ndarray) -> np.ndarray:
    """Row i (all heads) attends to keys [0, limits[i]) of K, V [keys, Hkv, Dh]
    (query head h uses K/V head h // (H / Hkv)).

    Rows that share a key limit are evaluated together, a few hundred at a time,
    as per-head matrix products (scores [H, rows, keys], softmax over keys, then
    the weighted sum of V): the same formula as one row at a time."""
    n, H, dh = q.shape
    out = np.zeros_like(q)
    scale = 1.0 / np.sqrt(dh)
    limits = np.asarray(limits)
    for lim in np.unique(limits):
        lim = int(lim)
        rows = np.flatnonzero(limits == lim)
        k = group_heads(K[:lim], H).transpose(1, 2, 0)      # [H, Dh, lim]
        v = group_heads(V[:lim], H).transpose(1, 0, 2)      # [H, lim, Dh]
        for c0 in range(0, len(rows), 256):
            r = rows[c0:c0 + 256]
            s = np.matmul(q[r].transpose(1, 0, 2), k) * scale   # [H, rows, lim]
            p = softmax(s)
            out[r] = np.matmul(p, v).transpose(1, 0, 2)         # [rows, H, Dh]
    return out


def attend_masked(q: np.ndarray, K: np.ndarray, V: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """Row i attends to the keys j with allowed[i, j] (explicit boolean mask)."""
    n, H, dh = q.shape
    out = np.zeros_like(q)
    scale = 1.0 / np.sqrt(dh)
    Kg, Vg = group_heads(K, H), group_heads(V, H)
    for i in range(n):
        idx = np.nonzero(allowed[i])[0]
        s = np.einsum("hd,khd->hk", q[i], Kg[idx]) * scale
        p = softmax(s)
        out[i] = np.einsum("hk,khd->hd", p, Vg[idx])
    return out


def confidence(logits: np.ndarray):
    """(argmax id with lowest-id ties, softmax probability of that id) per row.

    conf = 1 / sum_v exp(l_v - l_max); entries at -inf (the MASK id) add 0.
    """
    ids = np.argmax(logits, axis=-1).astype(np.int32)
    m = logits[np.arange(logits.shape[0]), ids][:, None]
    conf = 1.0 / np.sum(np.exp(logits - m), axis=-1)
    return ids, conf


# -----------------------------------------------------------------------------
# int8 weights (per-output-row scales)
# -----------------------------------------------------------------------------


def quantize_rows_int8(w: np.ndarray):
    """Symmetric per-row int8 quantisation, decided in float32.

    s[n] = max_k |w[n,k]| / 127 and q = clamp(round_half_even(w / s), -127, 127),
    both divisions in IEEE float32.  A zero row gets s = 0 and q = 0.
    Returns (q int8 [N,K], s float32 [N]).
    """
    w = np.asarray(w, dtype=np.float32)
    amax = np.max(np.abs(w), axis=1)
    s = (amax / np.float32(127.0)).astype(np.float32)
    safe = np.where(s > 0, s, np.float32(1.0)).astype(np.float32)
    q = np.rint(w / safe[:, None]).astype(np.float32)
    q = np.clip(q, -127, 127)
    q[s == 0] = 0
    return q.astype(np.int8), s


def dequantize_rows(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    return q.astype(np.float64) * s.astype(np.float64)[:, None]


# -----------------------------------------------------------------------------
# Q4_0 weights (Implementation section: the operator library's Q4_0 matrix
# multiplication; Evaluation: all models run Q4_0).  The GGUF Q4_0 format: each
# row is cut into blocks of 32 consecutive input columns; a block stores one fp16
# scale d and 32 four-bit codes q in [0, 15]; a weight is (q - 8) * d.
# -----------------------------------------------------------------------------

Q4_BLOCK = 32


def quantize_rows_q4_0(w: np.ndarray):
    """Q4_0 quantisation of every row of w [N, K], decided in float32.

    Per block: m = the block's value of largest magnitude (the first one in column
    order on ties), keeping its sign; d = m / -8; id = 1 / d (0 if d = 0);
    q = min(15, trunc(x * id + 8.5)) for every x of the block; the stored scale is
    d rounded to fp16 (round to nearest even).  A ragged last block (K not a
    multiple of 32) is padded with zeros.  Returns (q uint8 [N, nb*32], d float16
    [N, nb]), nb = ceil(K / 32)."""
    w = np.asarray(w, dtype=np.float32)
    N, K = w.shape
    nb = -(-K // Q4_BLOCK)
    x = np.zeros((N, nb * Q4_BLOCK), np.float32)
    x[:, :K] = w
    x = x.reshape(N, nb, Q4_BLOCK)
    first_max = np.argmax(np.abs(x), axis=2)                       # first index of max |x|
    m = np.take_along_axis(x, first_max[:, :, None], axis=2)[:, :, 0]
    d = (m / np.float32(-8.0)).astype(np.float32)
    with np.errstate(divide="ignore"):
        inv = np.where(d != 0, np.float32(1.0) / np.where(d != 0, d, np.float32(1.0)), np.float32(0.0))
    inv = inv.astype(np.float32)
    v = (x * inv[:, :, None]).astype(np.float32) + np.float32(8.5)   # float32 product, then float32 sum
    q = np.minimum(np.trunc(v.astype(np.float32)), 15).astype(np.uint8)
    return q.reshape(N, nb * Q4_BLOCK), d.astype(np.float16)


def dequantize_q4_0(q: np.ndarray, d: np.ndarray, K: int) -> np.ndarray:
    """Weights (q - 8) * d in float64, the padding columns dropped."""
    N, nb = d.shape
    w = (q.reshape(N, nb, Q4_BLOCK).astype(np.float64) - 8.0) * d.astype(np.float64)[:, :, None]
    return w.reshape(N, nb * Q4_BLOCK)[:, :K]


# -----------------------------------------------------------------------------
# Model parameters
# -----------------------------------------------------------------------------


GEMM_WEIGHTS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
QKV_BIASES = ("bq", "bk", "bv")


def _f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:                       # bfloat16 bit patterns: exact widening
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


class OracleModel:
    """Parameters in float64.

    `weights` is the dict written by ``synth.all_weights`` (float32 or bfloat16
    bit patterns), or a callable ``layer -> per-layer dict`` plus the globals, so
    that very large models can be materialised one layer at a time.
    With ``int8=True`` every matrix except the embedding is replaced by its
    dequantised int8 form q * s (per output row); with ``q4=True`` by its
    dequantised Q4_0 form (q - 8) * d (per row and 32-column block).
    """

    def __init__(self, shape, weights: dict, int8: bool = False, cache_layers: Optional[bool] = None,
                 layer_source=None, q4: bool = False):
        assert not (int8 and q4)
        self.shape = shape
        self.int8 = int8
        self.q4 = q4
        self._src = weights
        self._layer_source = layer_source
        if cache_layers is None:
            cache_layers = shape.params_per_layer * shape.n_layers * 8 < (2 << 30)
        self._cache = {} if cache_layers else None
        self.embed = _f64(weights["embed"])
        self.final_norm = _f64(weights["final_norm"])
        self._lm_src = weights["lm_head"]
        self._lm = None
        if self._cache is not None or int8 or q4:
            self._lm = self._convert_matrix(self._lm_src)

    def _convert_matrix(self, w):
        if self.int8 or self.q4:
            wf = w if w.dtype == np.float32 else (w.astype(np.uint32) << 16).view(np.float32)
            if self.q4:
                q, d = quantize_rows_q4_0(wf)
                return dequantize_q4_0(q, d, wf.shape[1])
            q, s = quantize_rows_int8(wf)
            return dequantize_rows(q, s)
        return _f64(w)

    def layer(self, l: int) -> dict:
        if self._cache is not None and l in self._cache:
            return self._cache[l]
        src = self._layer_source(l) if self._layer_source is not None else self._src["layers"][l]
        out = {k: self._convert_matrix(src[k]) for k in GEMM_WEIGHTS}
        for b in QKV_BIASES:      # Q/K/V biases (fp32, never quantised); zero when absent
            out[b] = _f64(src[b]) if b in src else 0.0
        out["attn_norm"] = _f64(src["attn_norm"])
        out["ffn_norm"] = _f64(src["ffn_norm"])
        if self._cache is not None:
            self._cache[l] = out
        return out

    def lm_logits(self, hf: np.ndarray, chunk: int = 16384) -> np.ndarray:
        """hf @ W_lm^T, with the MASK column set to -inf."""
        V = self.shape.vocab
        out = np.empty((hf.shape[0], V), np.float64)
        if self._lm is not None:
            out[:] = hf @ self._lm.T
        else:
            for b in range(0, V, chunk):
                e = min(V, b + chunk)
                out[:, b:e] = hf @ _f64(self._lm_src[b:e]).T
        out[:, self.shape.mask_id] = NEG_INF
        return out


# -----------------------------------------------------------------------------
# Prefix KV cache
# -----------------------------------------------------------------------------


class OracleKV:
    """Per-layer K and V (after RoPE for K) of every cached position, float64,
    [layer, position, K/V head, dim].

    fp16=True stores every K/V value rounded to IEEE half precision (round to
    nearest even), the paper's FP16 KV states (Implementation); the default keeps
    them exact.  (Values past the half range would become infinite here; the tests
    keep K and V far inside it.)"""

    def __init__(self, shape, capacity: int, fp16: bool = False):
        L, H, dh = shape.n_layers, shape.kv_heads, shape.head_dim
        self.shape = shape
        self.capacity = capacity
        self.fp16 = fp16
        self.K = np.zeros((L, capacity, H, dh))
        self.V = np.zeros((L, capacity, H, dh))
        self.prefix_len = 0
        self.prompt_len = 0

    def store(self, layer: int, pos: np.ndarray, k: np.ndarray, v: np.ndarray) -> None:
        if self.fp16:
            k = k.astype(np.float16).astype(np.float64)
            v = v.astype(np.float16).astype(np.float64)
        self.K[layer, pos] = k
        self.V[layer, pos] = v

    def copy(self) -> "OracleKV":
        c = OracleKV.__new__(OracleKV)
        c.shape, c.capacity, c.fp16 = self.shape, self.capacity, self.fp16
        c.K, c.V = self.K.copy(), self.V.copy()
        c.prefix_len, c.prompt_len = self.prefix_len, self.prompt_len
        return c

    def block_of(self, p: int) -> int:
        """Block index: 0 for prompt positions, 1 + (p - P0) // block after it."""
        if p < self.prompt_len:
            return 0
        return 1 + (p - self.prompt_len) // self.shape.block

    def end_of_block(self, p: int) -> int:
        b = self.block_of(p)
        end = self.prompt_len + self.shape.block * b
        return min(end, self.prefix_len)


# -----------------------------------------------------------------------------
# Forward over a query set with a prefix cache
# -----------------------------------------------------------------------------


def forward_rows(model: OracleModel, kv: OracleKV, ids: np.ndarray, pos: np.ndarray,
                 limits: np.ndarray, lm_head: bool, stop_layer: Optional[int] = None):
    """Run the rows (ids at absolute positions pos) through every layer.

    At each layer the rows' K/V are written into the cache at their positions
    first, then row i attends to cache keys [0, limits[i]).  Returns the
    residual stream x [n, d] and, if lm_head, the logits [n, V].
    """
    sh = model.shape
    n = len(ids)
    H, Hkv, dh = sh.n_heads, sh.kv_heads, sh.head_dim
    pos = np.asarray(pos, dtype=np.int64)
    x = model.embed[np.asarray(ids, dtype=np.int64)].copy()
    n_layers = sh.n_layers if stop_layer is None else stop_layer
    for l in range(n_layers):
        w = model.layer(l)
        h = rmsnorm(x, w["attn_norm"], sh.eps)
        q = (h @ w["wq"].T + w["bq"]).reshape(n, H, dh)
        k = (h @ w["wk"].T + w["bk"]).reshape(n, Hkv, dh)
        v = (h @ w["wv"].T + w["bv"]).reshape(n, Hkv, dh)
        q = rope(q, pos, sh.rope_base)
        k = rope(k, pos, sh.rope_base)
        kv.store(l, pos, k, v)
        o = attend(q, kv.K[l], kv.V[l], limits)
        x = x + o.reshape(n, H * dh) @ w["wo"].T
        h2 = rmsnorm(x, w["ffn_norm"], sh.eps)
        x = x + (silu(h2 @ w["wg"].T) * (h2 @ w["wu"].T)) @ w["wd"].T
    logits = None
    if lm_head and stop_layer is None:
        logits = model.lm_logits(rmsnorm(x, model.final_norm, sh.eps))
    return x, logits


def input_ids(shape, tok: np.ndarray, mask: np.ndarray) -> np.ndarray:
    """Token fed to the model: the MASK id where the mask flag is set."""
    return np.where(np.asarray(mask) != 0, shape.mask_id, np.asarray(tok)).astype(np.int32)


def prefill(model: OracleModel, kv: OracleKV, prompt: np.ndarray) -> None:
    """Prompt processing: the prompt is one bidirectional block at positions [0, P0)."""
    n = len(prompt)
    assert kv.prefix_len == 0 and n <= kv.capacity
    forward_rows(model, kv, prompt, np.arange(n), np.full(n, n), lm_head=False)
    kv.prefix_len = n
    kv.prompt_len = n


@dataclasses.dataclass
class StepOut:
    logits: np.ndarray
    ids: np.ndarray
    conf: np.ndarray
    x: np.ndarray


def denoise_step(model: OracleModel, kv: OracleKV, tok: np.ndarray, mask: np.ndarray) -> StepOut:
    """One denoising step over the window rows at [P, P + W).

    Every window row attends to all keys [0, P + W): the whole prefix plus the
    window itself, bidirectionally (current block and any draft block alike).
    The prefix length is unchanged; the window's K/V land in rows [P, P + W),
    which are scratch until a block is appended.
    """
    W = len(tok)
    P = kv.prefix_len
    assert P + W <= kv.capacity
    ids = input_ids(model.shape, tok, mask)
    x, logits = forward_rows(model, kv, ids, P + np.arange(W), np.full(W, P + W), lm_head=True)
    ids_out, conf = confidence(logits)
    return StepOut(logits, ids_out, conf, x)


def denoise_window(model: OracleModel, kv: OracleKV, w0: int, tok: np.ndarray, mask: np.ndarray) -> StepOut:
    """One denoising step over a decoding window at [w0, w0 + W) with w0 >= P
    (System Design, "Multi-Block Speculative Decoding": the window is the execution
    unit and slides along the commit frontier).  Rows [P, w0) are committed
    positions the window has slid past: their cached K/V are the ones an earlier
    window step wrote and are reused as they are.  Window rows attend to every key in
    [0, w0 + W); their K/V land in rows [w0, w0 + W).  With w0 = P this is
    denoise_step."""
    W = len(tok)
    assert kv.prefix_len <= w0 and w0 + W <= kv.capacity
    ids = input_ids(model.shape, tok, mask)
    x, logits = forward_rows(model, kv, ids, w0 + np.arange(W), np.full(W, w0 + W), lm_head=True)
    ids_out, conf = confidence(logits)
    return StepOut(logits, ids_out, conf, x)


def skip_logits(out: StepOut, need: Optional[np.ndarray], n_need: int):
    """Selective logits skipping (System Design, "Dual-Path Progressive Revision",
    "Selective Logits Skipping"): the output projection, the confidence and the
    selection run only for positions whose identity or confidence can still matter;
    the other positions are skipped.  `need` flags those rows (None: every row);
    at most n_need of them are evaluated, the first ones in row order.  A skipped
    row reports id -1 and confidence 0.  Returns (ids, conf)."""
    W = len(out.ids)
    flag = np.ones(W, dtype=bool) if need is None else (np.asarray(need) != 0)
    chosen = np.zeros(W, dtype=bool)
    chosen[np.flatnonzero(flag)[:max(0, n_need)]] = True
    ids = np.where(chosen, out.ids, -1).astype(np.int64)
    conf = np.where(chosen, out.conf, 0.0)
    return ids, conf


def denoise_window_sls(model: OracleModel, kv: OracleKV, w0: int, tok: np.ndarray, mask: np.ndarray,
                       need: Optional[np.ndarray], n_need: int):
    """denoise_window with selective logits skipping: the forward (and the K/V it
    writes) is the window step's; only the rows skip_logits keeps get an output."""
    out = denoise_window(model, kv, w0, tok, mask)
    ids, conf = skip_logits(out, need, n_need)
    return ids, conf, out


def commit(conf: np.ndarray, pred: np.ndarray, tok: np.ndarray, mask: np.ndarray,
           seg_begin: int, seg_len: int, k: int):
    """Commit the k most confident masked positions of [seg_begin, seg_begin + seg_len).

    Order: higher confidence first, equal confidence -> lower position.  The
    chosen positions take their predicted id and leave the mask.  Returns the
    committed positions in that order (min(k, #masked) of them).
    """
    cand = [p for p in range(seg_begin, seg_begin + seg_len) if mask[p]]
    cand.sort(key=lambda p: (-float(conf[p]), p))
    chosen = cand[:max(0, k)]
    for p in chosen:
        tok[p] = pred[p]
        mask[p] = 0
    return np.array(chosen, dtype=np.int32)


def append_block(model: OracleModel, kv: OracleKV, block_tok: np.ndarray) -> None:
    """Append a completed block: its rows at [P, P + n) see keys [0, P + n)."""
    n = len(block_tok)
    P = kv.prefix_len
    assert P + n <= kv.capacity
    assert np.all(np.asarray(block_tok) != model.shape.mask_id)
    forward_rows(model, kv, block_tok, P + np.arange(n), np.full(n, P + n), lm_head=False)
    kv.prefix_len = P + n


def refresh(model: OracleModel, kv: OracleKV, pos: Sequence[int], new_ids: Sequence[int],
            lm_head: bool = True):
    """Sparse refresh of revised prefix positions.

    Each revised row is recomputed from its new id; at every layer its K/V
    replace the cached ones (all refreshed rows before that layer's attention),
    and it attends to keys [0, end of its block).  Every other cached row is left
    as it was.  Returns (ids, conf, logits) of the refreshed rows if lm_head.
    """
    pos = np.asarray(pos, dtype=np.int64)
    assert len(set(pos.tolist())) == len(pos)
    assert np.all(pos < kv.prefix_len)
    limits = np.array([kv.end_of_block(int(p)) for p in pos])
    x, logits = forward_rows(model, kv, np.asarray(new_ids), pos, limits, lm_head=lm_head)
    if not lm_head:
        return None
    ids, conf = confidence(logits)
    return ids, conf, logits


# Token states of staged stabilisation (System Design, "Staged Token Stabilization").
IV, V, S = 0, 1, 2      # invisible (masked), visible (exposed, still revisable), stable


def commit_staged(conf: np.ndarray, pred: np.ndarray, tok: np.ndarray, mask: np.ndarray, state: np.ndarray,
                  seg_begin: int, seg_len: int, theta_visible: float, theta_stable: float):
    """One step of staged token stabilisation over [seg_begin, seg_begin + seg_len)
    (System Design, "Staged Token Stabilization"; thresholds 0.7 / 0.9 in the Evaluation
    setup).

    - Every invisible position whose confidence reaches theta_visible becomes visible:
      it takes its predicted id and leaves the mask.
    - If none did and invisible positions remain, the most confident of them becomes
      visible (equal confidence -> lower position), so that decoding always progresses.
    - Every visible position, the ones just promoted included, whose held token passes
      the stability criterion becomes stable: this step predicts the id the position
      holds (pred == tok) with a confidence that reaches theta_stable.  Stability is a
      property of the held token; a row whose prediction moved to another id, however
      confidently, stays visible and tracked.  For theta_stable > 1/2 this is exactly
      "the held token's own probability reaches theta_stable", since a token other
      than the argmax has probability at most 1 - conf < 1/2.  A visible position keeps
      its id here: identity revision of visible tokens goes through the refresh path.

    Confidences and thresholds are compared in float32 (the precision the confidence
    is produced in).  Returns the positions that left the invisible state, ascending.
    """
    c = np.asarray(conf, dtype=np.float32)
    tv, ts = np.float32(theta_visible), np.float32(theta_stable)
    seg = range(seg_begin, seg_begin + seg_len)
    cand = [p for p in seg if state[p] == IV]
    promoted = [p for p in cand if c[p] >= tv]
    if not promoted and cand:
        promoted = [min(cand, key=lambda p: (-float(c[p]), p))]
    for p in promoted:
        tok[p] = pred[p]
        mask[p] = 0
        state[p] = V
    for p in seg:
        if state[p] == V and c[p] >= ts and pred[p] == tok[p]:
            state[p] = S
    return np.array(sorted(promoted), dtype=np.int32)


def repredict_tracked(model: OracleModel, kv: OracleKV, tracked: dict, theta_visible: float,
                      theta_stable: float):
    """Re-prediction of the visible tokens that stay tracked after their block entered
    the prefix (System Design, "Staged Token Stabilization": visible tokens remain
    tracked until they pass the stability threshold; "Sparse Cache Refresh": their
    confidence, identity and KV are recomputed sparsely and merged before the next
    step).

    `tracked` maps a prefix position to the id it holds.  The tracked positions are
    taken block by block, in block order.  For block b:
      1. every tracked position of b is recomputed at once as MASK (one sparse refresh:
         their K/V replace the cached ones layer by layer, each row attends to the keys
         up to the end of its block), which gives the model's (id, conf) for it with
         the block's other tracked tokens hidden and everything else as it stands;
      2. per position, in float32: conf >= theta_stable -> the new id, and the position
         becomes stable (no longer tracked); conf >= theta_visible -> the new id, still
         visible; otherwise it keeps its id;
      3. the chosen ids of block b are written back with a second sparse refresh, so
         the cache holds their K/V before block b + 1 is re-predicted.
    The result depends only on the tracked set and the cache, not on how many rows
    one call may carry.  Updates `tracked` in place; returns (positions that became
    stable, ascending; {position: id written back})."""
    tv, ts = np.float32(theta_visible), np.float32(theta_stable)
    mask_id = model.shape.mask_id
    stable, chosen = [], {}
    for b in sorted({kv.block_of(int(p)) for p in tracked}):
        pos = sorted(int(p) for p in tracked if kv.block_of(int(p)) == b)
        ids, conf, _ = refresh(model, kv, pos, [mask_id] * len(pos))
        new = []
        for j, p in enumerate(pos):
            c = np.float32(conf[j])
            if c >= ts:
                new.append(int(ids[j]))
                stable.append(p)
            elif c >= tv:
                new.append(int(ids[j]))
            else:
                new.append(int(tracked[p]))
        refresh(model, kv, pos, new, lm_head=False)
        for p, t in zip(pos, new):
            chosen[p] = t
            tracked[p] = t
    for p in stable:
        del tracked[p]
    return sorted(stable), chosen


def commit_schedule(n_masked: int, steps: int) -> list:
    """Commits per step: floor(N / s) + [t < N mod s] for t = 0 .. s-1."""
    base, rem = divmod(n_masked, steps)
    return [base + (1 if t < rem else 0) for t in range(steps)]


# -----------------------------------------------------------------------------
# Brute force: one forward of a whole sequence under an explicit mask
# -----------------------------------------------------------------------------


def block_causal_allowed(n_total: int, prompt_len: int, block: int, window_from: Optional[int] = None):
    """allowed[i, j]: prompt = block 0 (bidirectional); block b sees blocks <= b.

    Rows at or after `window_from` (a denoising window) see every row.
    """
    b = np.array([0 if j < prompt_len else 1 + (j - prompt_len) // block for j in range(n_total)])
    allowed = b[None, :] <= b[:, None]
    if window_from is not None:
        allowed[window_from:, :] = True
    return allowed


def forward_full(model: OracleModel, ids: np.ndarray, allowed: np.ndarray):
    """Recompute every row from scratch (no cache) under the boolean mask.

    Returns (x [n, d], logits [n, V], K [L, n, Hkv, Dh], V [L, n, Hkv, Dh]).
    """
    sh = model.shape
    n = len(ids)
    H, Hkv, dh = sh.n_heads, sh.kv_heads, sh.head_dim
    pos = np.arange(n)
    x = model.embed[np.asarray(ids, dtype=np.int64)].copy()
    Ks, Vs = [], []
    for l in range(sh.n_layers):
        w = model.layer(l)
        h = rmsnorm(x, w["attn_norm"], sh.eps)
        q = rope((h @ w["wq"].T + w["bq"]).reshape(n, H, dh), pos, sh.rope_base)
        k = rope((h @ w["wk"].T + w["bk"]).reshape(n, Hkv, dh), pos, sh.rope_base)
        v = (h @ w["wv"].T + w["bv"]).reshape(n, Hkv, dh)
        Ks.append(k)
        Vs.append(v)
        o = attend_masked(q, k, v, allowed)
        x = x + o.reshape(n, H * dh) @ w["wo"].T
        h2 = rmsnorm(x, w["ffn_norm"], sh.eps)
        x = x + (silu(h2 @ w["wg"].T) * (h2 @ w["wu"].T)) @ w["wd"].T
    logits = model.lm_logits(rmsnorm(x, model.final_norm, sh.eps))
    return x, logits, np.stack(Ks), np.stack(Vs)
