"""Pins of the oracle against facts that do not come from the oracle itself.

Each test checks the float64 oracle against a closed form, an invariant, a
library routine (PyTorch functional ops, SciPy softmax), or brute force on tiny
inputs.  Together they are meant to catch a dropped term, a wrong sign or
index, or a transposed operand anywhere in the oracle.
"""
import dataclasses
import itertools
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import model as om

MICRO = synth.MICRO


def micro_model(shape=MICRO, seed=0, int8=False):
    w = synth.all_weights(shape, "f32", seed)
    return oracle.OracleModel(shape, w, int8=int8), w


# ----------------------------------------------------------------------------
# An independent reference: PyTorch functional ops, complex-number RoPE, SDPA
# ----------------------------------------------------------------------------


def torch_forward(shape, w, ids, allowed):
    """Full forward of a sequence (positions 0..n-1) under a boolean mask."""
    t = lambda a: torch.from_numpy(synth.as_f32(np.asarray(a))).double()
    n = len(ids)
    H, dh, d = shape.n_heads, shape.head_dim, shape.d_model
    Hkv = shape.kv_heads
    half = dh // 2
    pos = torch.arange(n, dtype=torch.float64)
    inv = shape.rope_base ** (-torch.arange(half, dtype=torch.float64) * 2.0 / dh)
    rot = torch.polar(torch.ones(n, half, dtype=torch.float64), pos[:, None] * inv)  # e^{i theta}

    def rope_c(u):  # u [n, H, dh]: pair (j, j + half) as the complex number u_j + i u_{j+half}
        z = torch.complex(u[..., :half], u[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    x = t(w["embed"])[torch.as_tensor(np.asarray(ids, np.int64))]
    mask = torch.as_tensor(allowed)
    for lw in w["layers"]:
        b = {k: (t(lw[k]) if k in lw else None) for k in ("bq", "bk", "bv")}
        h = F.rms_norm(x, (d,), weight=t(lw["attn_norm"]), eps=shape.eps)
        q = rope_c(F.linear(h, t(lw["wq"]), b["bq"]).view(n, H, dh))
        k = rope_c(F.linear(h, t(lw["wk"]), b["bk"]).view(n, Hkv, dh))
        v = F.linear(h, t(lw["wv"]), b["bv"]).view(n, Hkv, dh)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           attn_mask=mask, enable_gqa=Hkv != H)
        x = x + F.linear(o.transpose(0, 1).reshape(n, d), t(lw["wo"]))
        h2 = F.rms_norm(x, (d,), weight=t(lw["ffn_norm"]), eps=shape.eps)
        x = x + F.linear(F.silu(F.linear(h2, t(lw["wg"]))) * F.linear(h2, t(lw["wu"])), t(lw["wd"]))
    hf = F.rms_norm(x, (d,), weight=t(w["final_norm"]), eps=shape.eps)
    logits = F.linear(hf, t(w["lm_head"]))
    logits[:, shape.mask_id] = -float("inf")
    return logits.numpy()


# ----------------------------------------------------------------------------
# Operators: closed forms and special cases
# ----------------------------------------------------------------------------


def test_rmsnorm_constant_vector_is_gain():
    g = np.linspace(0.5, 2.0, 16)
    for c in (3.0, -0.25, 1e3):
        out = oracle.rmsnorm(np.full((1, 16), c), g, 1e-5)
        np.testing.assert_allclose(out[0], g * c / np.sqrt(c * c + 1e-5), rtol=1e-14)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x, g = rng.normal(size=(5, 48)), rng.normal(size=48)
    ref = F.rms_norm(torch.from_numpy(x), (48,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref, rtol=1e-12, atol=1e-14)


def test_rope_identity_at_position_zero():
    u = np.random.default_rng(1).normal(size=(3, 2, 8))
    np.testing.assert_array_equal(oracle.rope(u, np.zeros(3, np.int64), 10000.0), u)


def test_rope_is_complex_rotation_and_relative():
    rng = np.random.default_rng(2)
    dh, base = 16, 10000.0
    q, k = rng.normal(size=(1, 1, dh)), rng.normal(size=(1, 1, dh))
    # complex form: z_j = u_j + i u_{j+dh/2} multiplied by exp(i * pos * base^(-2j/dh))
    half = dh // 2
    ang = 7 * base ** (-2.0 * np.arange(half) / dh)
    z = (q[0, 0, :half] + 1j * q[0, 0, half:]) * np.exp(1j * ang)
    r = oracle.rope(q, np.array([7]), base)[0, 0]
    np.testing.assert_allclose(r, np.concatenate([z.real, z.imag]), rtol=1e-13, atol=1e-15)
    # norm preserved, and q.k depends only on the position difference
    assert np.isclose(np.linalg.norm(r), np.linalg.norm(q), rtol=1e-13)
    d1 = np.sum(oracle.rope(q, np.array([11]), base) * oracle.rope(k, np.array([4]), base))
    d2 = np.sum(oracle.rope(q, np.array([107]), base) * oracle.rope(k, np.array([100]), base))
    assert np.isclose(d1, d2, rtol=1e-10)


def test_attention_uniform_when_scores_vanish():
    rng = np.random.default_rng(3)
    V = rng.normal(size=(9, 2, 4))
    q = np.zeros((3, 2, 4))
    out = oracle.attend(q, rng.normal(size=(9, 2, 4)), V, np.array([9, 5, 1]))
    np.testing.assert_allclose(out[0], V.mean(axis=0), rtol=1e-13)
    np.testing.assert_allclose(out[1], V[:5].mean(axis=0), rtol=1e-13)
    np.testing.assert_allclose(out[2], V[0], rtol=1e-13)


def test_attention_matches_sdpa():
    rng = np.random.default_rng(4)
    n, T, H, dh = 4, 11, 3, 8
    q, K, V = rng.normal(size=(n, H, dh)), rng.normal(size=(T, H, dh)), rng.normal(size=(T, H, dh))
    limits = np.array([11, 7, 3, 1])
    allowed = np.arange(T)[None, :] < limits[:, None]
    ref = F.scaled_dot_product_attention(torch.from_numpy(q).transpose(0, 1),
                                         torch.from_numpy(K).transpose(0, 1),
                                         torch.from_numpy(V).transpose(0, 1),
                                         attn_mask=torch.from_numpy(allowed)).transpose(0, 1).numpy()
    np.testing.assert_allclose(oracle.attend(q, K, V, limits), ref, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(oracle.attend_masked(q, K, V, allowed), ref, rtol=1e-11, atol=1e-13)


def test_silu_closed_form():
    z = np.array([-3.0, 0.0, 0.5, 10.0])
    np.testing.assert_allclose(oracle.silu(z), z * scipy.special.expit(z), rtol=1e-14)


def test_confidence_is_softmax_max_without_mask():
    rng = np.random.default_rng(5)
    logits = rng.normal(size=(6, 50)) * 2
    logits[:, 49] = -np.inf
    logits[2, 10] = logits[2, 3] = 100.0          # a tie: lowest id wins
    ids, conf = oracle.confidence(logits)
    p = scipy.special.softmax(logits, axis=-1)
    assert np.all(ids != 49)
    assert ids[2] == 3
    np.testing.assert_array_equal(ids, np.argmax(p, axis=-1))
    np.testing.assert_allclose(conf, p.max(axis=-1), rtol=1e-13)
    np.testing.assert_allclose(p.sum(axis=-1), 1.0, rtol=1e-13)


def test_planted_lm_head_row_forces_argmax():
    sh = MICRO
    model, _ = micro_model()
    hf = oracle.rmsnorm(np.random.default_rng(6).normal(size=(1, sh.d_model)), model.final_norm, sh.eps)
    alpha, t = 0.05, 17
    model._lm = model._lm.copy()
    model._lm[t] = alpha * hf[0]
    logits = model.lm_logits(hf)
    ids, conf = oracle.confidence(logits)
    assert ids[0] == t
    expect = 1.0 / np.sum(np.exp(np.delete(logits[0], sh.mask_id) - alpha * hf[0] @ hf[0]))
    np.testing.assert_allclose(conf[0], expect, rtol=1e-12)


# ----------------------------------------------------------------------------
# The whole forward against the independent PyTorch reference
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("shape", [MICRO, synth.TINY.with_layers(1), synth.MICRO_GQA,
                                   synth.SMALL_MQA.with_layers(1)], ids=["micro", "tiny1", "micro_gqa", "small_mqa1"])
def test_step_matches_torch_reference(shape):
    model, w = micro_model(shape)
    P0, W = 24, 12
    prompt = synth.prompt_ids(shape, P0)
    kv = oracle.OracleKV(shape, P0 + W)
    oracle.prefill(model, kv, prompt)
    tok, mask = synth.window(shape, W, range(3, W))
    out = oracle.denoise_step(model, kv, tok, mask)
    seq = np.concatenate([prompt, oracle.input_ids(shape, tok, mask)])
    allowed = oracle.block_causal_allowed(P0 + W, P0, shape.block, window_from=P0)
    ref = torch_forward(shape, w, seq, allowed)[P0:]
    fin = np.isfinite(ref)
    np.testing.assert_array_equal(fin, np.isfinite(out.logits))
    np.testing.assert_allclose(out.logits[fin], ref[fin], rtol=1e-9, atol=1e-11)


def test_one_row_no_prefix_is_textbook_mlp_block():
    """A single row attends only to itself, so attention returns v."""
    sh = MICRO.with_layers(1)
    model, w = micro_model(sh)
    kv = oracle.OracleKV(sh, 4)
    ids = np.array([5])
    x, _ = oracle.forward_rows(model, kv, ids, np.array([0]), np.array([1]), lm_head=False)
    lw = {k: synth.as_f32(v).astype(np.float64) for k, v in w["layers"][0].items()}
    x0 = synth.as_f32(w["embed"])[5].astype(np.float64)
    h = x0 / np.sqrt(np.mean(x0 ** 2) + sh.eps) * lw["attn_norm"]
    x1 = x0 + lw["wo"] @ (lw["wv"] @ h)
    h2 = x1 / np.sqrt(np.mean(x1 ** 2) + sh.eps) * lw["ffn_norm"]
    g = lw["wg"] @ h2
    x2 = x1 + lw["wd"] @ (g / (1 + np.exp(-g)) * (lw["wu"] @ h2))
    np.testing.assert_allclose(x[0], x2, rtol=1e-12, atol=1e-14)


def test_gqa_equals_mha_with_each_kv_head_repeated():
    """Grouped-query attention is multi-head attention whose K/V projections give
    every query head of a group the same K/V head: repeating each K/V head's rows
    (and biases) G times must reproduce the grouped model exactly."""
    g = synth.MICRO_GQA
    G = g.n_heads // g.kv_heads
    m = dataclasses.replace(g, n_kv_heads=0)
    model_g, w = micro_model(g)
    wm = dict(w, layers=[])
    for lw in w["layers"]:
        lw2 = dict(lw)
        for name in ("wk", "wv", "bk", "bv"):
            a = lw[name].reshape(g.kv_heads, g.head_dim, *lw[name].shape[1:])
            lw2[name] = np.repeat(a, G, axis=0).reshape(g.d_model, *lw[name].shape[1:])
        wm["layers"].append(lw2)
    model_m = oracle.OracleModel(m, wm)
    P0, W = 24, 12
    prompt = synth.prompt_ids(g, P0)
    tok, mask = synth.window(g, W, range(3, W))
    outs = []
    for mod, sh in ((model_g, g), (model_m, m)):
        kv = oracle.OracleKV(sh, P0 + W)
        oracle.prefill(mod, kv, prompt)
        outs.append(oracle.denoise_step(mod, kv, tok, mask))
    fin = np.isfinite(outs[0].logits)
    np.testing.assert_allclose(outs[0].logits[fin], outs[1].logits[fin], rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------
# Cache = brute-force recompute (block-causal), step = full forward
# ----------------------------------------------------------------------------


def _build_prefix(model, sh, P0, n_blocks, cap):
    kv = oracle.OracleKV(sh, cap)
    prompt = synth.prompt_ids(sh, P0)
    oracle.prefill(model, kv, prompt)
    blocks = []
    for b in range(n_blocks):
        blk = synth.uniform_ids(50 + b, 1, sh.block, sh.mask_id)
        oracle.append_block(model, kv, blk)
        blocks.append(blk)
    return kv, np.concatenate([prompt] + blocks)


@pytest.mark.parametrize("sh", [MICRO, synth.MICRO_GQA], ids=["mha", "gqa"])
def test_cached_prefix_equals_block_causal_recompute(sh):
    model, _ = micro_model(sh)
    P0 = 20
    kv, seq = _build_prefix(model, sh, P0, 2, P0 + 2 * sh.block)
    _, _, K, V = oracle.forward_full(model, seq, oracle.block_causal_allowed(len(seq), P0, sh.block))
    np.testing.assert_allclose(kv.K[:, :len(seq)], K, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(kv.V[:, :len(seq)], V, rtol=1e-10, atol=1e-12)


def test_fp16_cache_stores_the_half_precision_rounding():
    """OracleKV(fp16=True) rounds at storage and nowhere else: layer 0's K/V depend
    only on the embeddings, so they are exactly numpy's round-to-nearest-even half
    values of the exact run's; every stored value is a half-precision number; later
    layers, which attend over the rounded cache, move by a small relative amount."""
    sh = MICRO
    model, _ = micro_model(sh)
    prompt = synth.prompt_ids(sh, 20)
    exact = oracle.OracleKV(sh, 20)
    half = oracle.OracleKV(sh, 20, fp16=True)
    oracle.prefill(model, exact, prompt)
    oracle.prefill(model, half, prompt)
    to_half = lambda a: a.astype(np.float16).astype(np.float64)
    np.testing.assert_array_equal(half.K[0], to_half(exact.K[0]))
    np.testing.assert_array_equal(half.V[0], to_half(exact.V[0]))
    np.testing.assert_array_equal(half.K, to_half(half.K))
    np.testing.assert_array_equal(half.V, to_half(half.V))
    d = np.abs(half.K[1] - exact.K[1]).max()
    assert 0 < d < 1e-2 * np.abs(exact.K[1]).max()
    assert half.copy().fp16


def test_block_mask_really_hides_the_future():
    """Changing a later block must not change earlier cached rows."""
    sh = MICRO
    model, _ = micro_model(sh)
    P0 = 20
    kv1, _ = _build_prefix(model, sh, P0, 1, P0 + 2 * sh.block)
    kv2 = kv1.copy()
    oracle.append_block(model, kv1, synth.uniform_ids(90, 1, sh.block, sh.mask_id))
    oracle.append_block(model, kv2, synth.uniform_ids(91, 1, sh.block, sh.mask_id))
    n = P0 + sh.block
    np.testing.assert_array_equal(kv1.K[:, :n], kv2.K[:, :n])
    assert not np.allclose(kv1.K[:, n:n + sh.block], kv2.K[:, n:n + sh.block])


def test_step_with_speculative_window_equals_full_forward():
    sh = MICRO
    model, _ = micro_model(sh)
    P0 = 20
    kv, seq = _build_prefix(model, sh, P0, 1, P0 + 3 * sh.block)
    W = 2 * sh.block
    tok, mask = synth.window(sh, W, list(range(24, 32)) + list(range(32, 64)))
    out = oracle.denoise_step(model, kv, tok, mask)
    full_seq = np.concatenate([seq, oracle.input_ids(sh, tok, mask)])
    allowed = oracle.block_causal_allowed(len(full_seq), P0, sh.block, window_from=len(seq))
    _, logits, _, _ = oracle.forward_full(model, full_seq, allowed)
    np.testing.assert_allclose(out.logits[:, :-1], logits[len(seq):, :-1], rtol=1e-10, atol=1e-12)
    assert kv.prefix_len == len(seq)            # a step never grows the prefix


def test_window_permutation_permutes_outputs():
    sh = MICRO
    model, _ = micro_model(sh)
    kv, seq = _build_prefix(model, sh, 16, 0, 16 + sh.block)
    P = kv.prefix_len
    ids = synth.uniform_ids(7, 1, sh.block, sh.vocab)
    pos = P + np.arange(sh.block)
    lim = np.full(sh.block, P + sh.block)
    perm = np.random.default_rng(8).permutation(sh.block)
    _, l1 = oracle.forward_rows(model, kv.copy(), ids, pos, lim, lm_head=True)
    _, l2 = oracle.forward_rows(model, kv.copy(), ids[perm], pos[perm], lim, lm_head=True)
    np.testing.assert_allclose(l2[:, :-1], l1[perm, :-1], rtol=1e-10, atol=1e-12)


# ----------------------------------------------------------------------------
# Selective logits skipping
# ----------------------------------------------------------------------------


def test_skip_logits_brute_force_over_every_need_mask():
    W = 5
    rng = np.random.default_rng(3)
    out = om.StepOut(logits=None, ids=rng.integers(0, 50, W), conf=rng.random(W), x=None)
    for bits in itertools.product([0, 1], repeat=W):
        need = np.array(bits, np.uint8)
        for n_need in range(W + 2):
            ids, conf = oracle.skip_logits(out, need, n_need)
            seen = 0
            for i in range(W):
                keep = bits[i] == 1 and seen < n_need
                seen += bits[i]
                assert ids[i] == (out.ids[i] if keep else -1)
                assert conf[i] == (out.conf[i] if keep else 0.0)
    ids, conf = oracle.skip_logits(out, None, W)
    np.testing.assert_array_equal(ids, out.ids)
    np.testing.assert_array_equal(conf, out.conf)
    ids, conf = oracle.skip_logits(out, None, 2)
    assert list(ids[2:]) == [-1] * (W - 2) and list(ids[:2]) == list(out.ids[:2])


def test_sls_window_is_full_forward_on_kept_rows_and_leaves_the_cache_as_the_step():
    sh = MICRO
    model, _ = micro_model(sh)
    P0 = 20
    kv, seq = _build_prefix(model, sh, P0, 1, P0 + 2 * sh.block)
    W = sh.block
    tok, mask = synth.window(sh, W, list(range(8, 32)))
    need = mask.copy()
    need[[9, 30]] = 0
    kv_full = kv.copy()
    P = kv.prefix_len
    ids, conf, _ = oracle.denoise_window_sls(model, kv, P, tok, mask, need, 15)
    oracle.denoise_window(model, kv_full, P, tok, mask)
    np.testing.assert_array_equal(kv.K, kv_full.K)
    np.testing.assert_array_equal(kv.V, kv_full.V)
    full_seq = np.concatenate([seq, oracle.input_ids(sh, tok, mask)])
    allowed = oracle.block_causal_allowed(len(full_seq), P0, sh.block, window_from=len(seq))
    _, logits, _, _ = oracle.forward_full(model, full_seq, allowed)
    ref_ids, ref_conf = oracle.confidence(logits[len(seq):])
    kept = np.flatnonzero(need)[:15]
    skipped = np.setdiff1d(np.arange(W), kept)
    np.testing.assert_array_equal(ids[kept], ref_ids[kept])
    np.testing.assert_allclose(conf[kept], ref_conf[kept], rtol=1e-10)
    assert np.all(ids[skipped] == -1) and np.all(conf[skipped] == 0.0)


# ----------------------------------------------------------------------------
# Refresh special cases
# ----------------------------------------------------------------------------


def test_refresh_with_unchanged_ids_is_noop():
    sh = MICRO
    model, _ = micro_model(sh)
    P0 = 20
    kv, seq = _build_prefix(model, sh, P0, 2, P0 + 2 * sh.block)
    before_K, before_V = kv.K.copy(), kv.V.copy()
    pos = np.array([P0 + 3, P0 + 40, 5])
    oracle.refresh(model, kv, pos, seq[pos], lm_head=False)
    np.testing.assert_allclose(kv.K, before_K, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(kv.V, before_V, rtol=1e-10, atol=1e-12)


def test_refresh_whole_last_block_equals_recompute():
    sh = MICRO
    model, _ = micro_model(sh)
    P0 = 20
    kv, seq = _build_prefix(model, sh, P0, 2, P0 + 2 * sh.block)
    last = np.arange(P0 + sh.block, P0 + 2 * sh.block)
    new = synth.uniform_ids(77, 1, sh.block, sh.mask_id)
    res = oracle.refresh(model, kv, last, new, lm_head=True)
    seq2 = seq.copy()
    seq2[last] = new
    _, logits, K, V = oracle.forward_full(model, seq2, oracle.block_causal_allowed(len(seq2), P0, sh.block))
    np.testing.assert_allclose(kv.K[:, :len(seq2)], K, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(kv.V[:, :len(seq2)], V, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(res[2][:, :-1], logits[last, :-1], rtol=1e-10, atol=1e-12)


def test_refresh_is_sparse():
    """Only the refreshed rows change; dependants keep their (stale) K/V."""
    sh = MICRO
    model, _ = micro_model(sh)
    P0 = 20
    kv, seq = _build_prefix(model, sh, P0, 2, P0 + 2 * sh.block)
    before = kv.K.copy()
    pos = np.array([P0 + 1, P0 + 33])
    oracle.refresh(model, kv, pos, np.array([1, 2]), lm_head=False)
    other = np.setdiff1d(np.arange(kv.prefix_len), pos)
    np.testing.assert_array_equal(kv.K[:, other], before[:, other])
    assert not np.allclose(kv.K[:, pos], before[:, pos])


# ----------------------------------------------------------------------------
# Commit and the generation loop
# ----------------------------------------------------------------------------


def test_commit_brute_force_exchange_property():
    rng = np.random.default_rng(9)
    for trial in range(200):
        n = int(rng.integers(1, 9))
        conf = rng.choice([0.1, 0.2, 0.3, 0.5], size=n)      # many ties
        mask = rng.integers(0, 2, size=n).astype(np.uint8)
        k = int(rng.integers(0, n + 2))
        tok = np.full(n, -1, np.int32)
        pred = np.arange(100, 100 + n, dtype=np.int32)
        m0 = mask.copy()
        chosen = oracle.commit(conf, pred, tok, mask, 0, n, k)
        masked = [p for p in range(n) if m0[p]]
        assert len(chosen) == min(k, len(masked))
        # brute force: the chosen set is the unique subset that beats every left-out candidate
        best = None
        for S in itertools.combinations(masked, len(chosen)):
            rest = [q for q in masked if q not in S]
            if all(conf[p] > conf[q] or (conf[p] == conf[q] and p < q) for p in S for q in rest):
                assert best is None
                best = set(S)
        assert set(chosen.tolist()) == best
        for p in chosen:
            assert tok[p] == pred[p] and mask[p] == 0
        assert np.all(mask[[q for q in range(n) if q not in chosen]] == m0[[q for q in range(n) if q not in chosen]])


def test_commit_segment_only():
    conf = np.array([0.9, 0.8, 0.7, 0.6])
    mask = np.ones(4, np.uint8)
    tok = np.zeros(4, np.int32)
    chosen = oracle.commit(conf, np.arange(4, dtype=np.int32) + 10, tok, mask, 2, 2, 1)
    assert chosen.tolist() == [2] and mask.tolist() == [1, 1, 0, 1]


@pytest.mark.parametrize("n,s", [(32, 4), (32, 32), (24, 7), (5, 8)])
def test_commit_schedule(n, s):
    k = oracle.commit_schedule(n, s)
    assert sum(k) == n and len(k) == s and max(k) - min(k) <= 1 and k == sorted(k, reverse=True)


def test_tiny_generation_invariants():
    """4 steps x top-8 over a 32-token all-MASK block (fp32 tiny model)."""
    sh = synth.TINY
    model, _ = micro_model(sh)
    kv = oracle.OracleKV(sh, 64 + 32)
    oracle.prefill(model, kv, synth.prompt_ids(sh, 64))
    tok, mask = synth.window(sh, 32, range(32))
    committed = {}
    for step, k in enumerate(oracle.commit_schedule(32, 4)):
        out = oracle.denoise_step(model, kv, tok, mask)
        p = scipy.special.softmax(out.logits, axis=-1)
        np.testing.assert_allclose(p.sum(axis=-1), 1.0, rtol=1e-12)
        np.testing.assert_allclose(out.conf, p.max(axis=-1), rtol=1e-12)
        assert np.all(out.ids != sh.mask_id)
        n_before = int(mask.sum())
        chosen = oracle.commit(out.conf, out.ids, tok, mask, 0, 32, k)
        assert len(chosen) == min(k, n_before) == 8
        for pos, t in committed.items():            # never re-masked, never changed
            assert mask[pos] == 0 and tok[pos] == t
        for pos in chosen:
            committed[int(pos)] = int(tok[pos])
        assert kv.prefix_len == 64
    assert mask.sum() == 0 and np.all(tok != sh.mask_id)


# ----------------------------------------------------------------------------
# int8 quantisation
# ----------------------------------------------------------------------------


def test_int8_quantiser_bounds():
    w = synth.as_f32(synth.weight(MICRO, "wg", 0, "bf16"))
    w[3] = 0.0
    q, s = oracle.quantize_rows_int8(w)
    assert q.dtype == np.int8 and s.dtype == np.float32
    assert np.all(np.abs(q.astype(int)) <= 127)
    nz = s > 0
    assert np.all(np.abs(q[nz]).max(axis=1) == 127)              # each row's extreme maps to 127
    assert np.all(q[3] == 0) and s[3] == 0
    err = np.abs(w.astype(np.float64) - oracle.dequantize_rows(q, s))
    assert np.all(err <= s[:, None].astype(np.float64) * (0.5 + 2e-5))   # w / s is itself rounded in float32


# Exact rational arithmetic: an IEEE float32 operation is the exact result rounded to
# 24 significant bits, ties to even (normal range).  These helpers state that rule with
# fractions.Fraction, independently of numpy's float32 arithmetic.
def _round_half_even(fr: Fraction) -> int:
    n = fr.numerator // fr.denominator
    r = fr - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return n


def _to_f32(fr: Fraction) -> Fraction:
    if fr == 0:
        return Fraction(0)
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    assert e >= -126, "subnormal results are not needed here"
    ulp = Fraction(2) ** (e - 23)
    return (1 if fr > 0 else -1) * _round_half_even(a / ulp) * ulp


def _int8_code_exact(w: float, amax: float) -> int:
    s = _to_f32(Fraction(amax) / 127)
    return max(-127, min(127, _round_half_even(_to_f32(Fraction(w) / s))))


def test_int8_quantiser_rounds_half_to_even():
    """A row whose extreme is 127 has the scale 1 exactly, so w / s = w: codes of
    values halfway between integers follow round-half-to-even.  Round-half-away
    would give 1, 3, -1, -3, 127 for the second, fourth, fifth, sixth and last
    entries."""
    w = np.array([[127.0, 0.5, 1.5, 2.5, -0.5, -2.5, 3.5, -126.5]], np.float32)
    q, s = oracle.quantize_rows_int8(w)
    assert s[0] == np.float32(1.0)
    assert q[0].tolist() == [127, 0, 2, 2, 0, -2, 4, -126]


def test_int8_quantiser_divides_in_float32():
    """Values next to a rounding boundary: the code is round-half-even of the
    float32-rounded quotient w / s, with s = float32(max|w| / 127).  The expected
    codes come from exact rational arithmetic.  Rows are built so that, for several
    entries, a float64 division (w / s in float64, or s itself kept in float64) would
    round to the other integer; the test requires that such entries exist."""
    rng = np.random.default_rng(11)
    rows, discriminating = [], 0
    for _ in range(60):
        amax = np.float32(rng.uniform(0.01, 0.1))
        s32 = np.float32(amax / np.float32(127))
        row = [amax]
        for k in rng.integers(-120, 120, 24):
            centre = np.float32((k + 0.5) * float(s32))
            w = centre
            for step in rng.integers(-3, 4, 1):
                for _ in range(abs(int(step))):
                    w = np.nextafter(w, np.float32(np.inf if step > 0 else -np.inf), dtype=np.float32)
            row.append(w)
            exact = _int8_code_exact(float(w), float(amax))
            via64 = int(np.clip(np.rint(float(w) / (float(amax) / 127.0)), -127, 127))
            via64s32 = int(np.clip(np.rint(float(w) / float(s32)), -127, 127))
            discriminating += int(exact != via64 or exact != via64s32)
        rows.append(row)
    w = np.array(rows, np.float32)
    q, s = oracle.quantize_rows_int8(w)
    for i in range(w.shape[0]):
        assert Fraction(float(s[i])) == _to_f32(Fraction(float(w[i, 0])) / 127)
        want = [_int8_code_exact(float(v), float(w[i, 0])) for v in w[i]]
        assert q[i].tolist() == want, i
    assert discriminating >= 20, discriminating


def test_int8_model_is_bf16_model_with_dequantised_weights():
    sh = MICRO
    w = synth.all_weights(sh, "bf16", 0)
    m8 = oracle.OracleModel(sh, w, int8=True)
    wd = dict(w)
    wd["lm_head"] = oracle.dequantize_rows(*oracle.quantize_rows_int8(synth.as_f32(w["lm_head"])))
    wd["layers"] = []
    for lw in w["layers"]:
        d = dict(lw)
        for k in om.GEMM_WEIGHTS:
            d[k] = oracle.dequantize_rows(*oracle.quantize_rows_int8(synth.as_f32(lw[k])))
        wd["layers"].append(d)
    mref = oracle.OracleModel(sh, wd)
    for m in (m8, mref):
        kv = oracle.OracleKV(sh, 40)
        oracle.prefill(m, kv, synth.prompt_ids(sh, 8))
        m.out = oracle.denoise_step(m, kv, *synth.window(sh, 32, range(32))).logits
    np.testing.assert_array_equal(m8.out, mref.out)


# ----------------------------------------------------------------------------
# Q4_0 weights
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_q4_0_recovers_representable_blocks_exactly(sign):
    """A block whose values are (c - 8) * d0 with a power-of-two d0 and at least one
    code 0 (the value -8 * d0 has the largest magnitude) quantises to exactly c and
    d0; with the block negated, d = -d0 and the codes are the same."""
    rng = np.random.default_rng(5)
    N, nb = 6, 5
    d0 = np.float32(2.0 ** -7)
    c = rng.integers(0, 16, (N, nb * 32))
    c[:, ::32] = 0                                     # a code 0 in every block
    x = ((c - 8) * d0 * sign).astype(np.float32)
    q, d = oracle.quantize_rows_q4_0(x)
    np.testing.assert_array_equal(q, c)
    np.testing.assert_array_equal(d.astype(np.float32), np.full((N, nb), d0 * sign, np.float32))
    np.testing.assert_array_equal(oracle.dequantize_q4_0(q, d, nb * 32), x.astype(np.float64))


def test_q4_0_error_bound_and_extreme_code():
    """|w - (q - 8) d| <= |d| / 2 (+ the fp16 rounding of d), except where the code
    clamps at 15 (w / d > 7.5), where it is <= |d|; the value of largest magnitude
    of every block gets code 0.  Ragged K pads the last block with zeros."""
    rng = np.random.default_rng(6)
    K = 32 * 7 + 13
    w = (rng.standard_normal((40, K)) * 0.02).astype(np.float32)
    w[3, 32:64] = 0.0                                  # an all-zero block: d = 0, codes 8
    q, d = oracle.quantize_rows_q4_0(w)
    deq = oracle.dequantize_q4_0(q, d, K)
    nb = d.shape[1]
    xp = np.zeros((40, nb * 32), np.float64)
    xp[:, :K] = w
    dd = np.repeat(d.astype(np.float64), 32, axis=1)
    d32 = np.repeat((np.max(np.abs(xp.reshape(40, nb, 32)), axis=2) / 8.0), 32, axis=1)   # |d| before fp16
    ratio = np.divide(xp, np.sign(dd) * d32, out=np.zeros_like(xp), where=d32 > 0)         # w / d
    bound = np.where(ratio > 7.5, 1.0, 0.5) * np.abs(dd) + 8.0 * np.abs(np.abs(dd) - d32) + 1e-12
    err = np.abs(xp - np.pad(deq, ((0, 0), (0, nb * 32 - K))))
    assert np.all(err <= bound)
    first = np.argmax(np.abs(xp.reshape(40, nb, 32)), axis=2)
    codes = q.reshape(40, nb, 32)
    nz = np.abs(d.astype(np.float64)) > 0
    assert np.all(np.take_along_axis(codes, first[:, :, None], axis=2)[:, :, 0][nz] == 0)
    assert np.all(q.reshape(40, nb, 32)[3, 1] == 8) and d[3, 1] == 0


def test_q4_0_sign_tie_goes_to_the_first_column():
    x = np.zeros((1, 32), np.float32)
    x[0, 4], x[0, 9] = 0.5, -0.5
    q, d = oracle.quantize_rows_q4_0(x)
    assert float(d[0, 0]) == -0.0625                   # m = +0.5 (column 4), d = m / -8
    assert q[0, 4] == 0 and q[0, 9] == 15 and q[0, 0] == 8
    np.testing.assert_array_equal(oracle.dequantize_q4_0(q, d, 32)[0, [4, 9]], [0.5, -0.4375])


def test_q4_0_model_is_bf16_model_with_dequantised_weights():
    sh = MICRO
    w = synth.all_weights(sh, "bf16", 0)
    m4 = oracle.OracleModel(sh, w, q4=True)
    deq = lambda a: oracle.dequantize_q4_0(*oracle.quantize_rows_q4_0(synth.as_f32(a)), a.shape[1])
    wd = dict(w)
    wd["lm_head"] = deq(w["lm_head"])
    wd["layers"] = []
    for lw in w["layers"]:
        dct = dict(lw)
        for k in om.GEMM_WEIGHTS:
            dct[k] = deq(lw[k])
        wd["layers"].append(dct)
    mref = oracle.OracleModel(sh, wd)
    for m in (m4, mref):
        kv = oracle.OracleKV(sh, 40)
        oracle.prefill(m, kv, synth.prompt_ids(sh, 8))
        m.out = oracle.denoise_step(m, kv, *synth.window(sh, 32, range(32))).logits
    np.testing.assert_array_equal(m4.out, mref.out)


def test_synth_inputs_are_reproducible_and_sliceable():
    a = synth.normal(0, 5, 1000, "bf16")
    b = synth.normal(0, 5, 101, "bf16", offset=333)
    np.testing.assert_array_equal(a[333:434], b)
    f = synth.as_f32(synth.normal(0, 6, 200000, "bf16"))
    assert abs(f.std() - 0.02) < 2e-4 and abs(f.mean()) < 2e-4
    ids = synth.prompt_ids(synth.TINY, 5000)
    assert ids.min() >= 0 and ids.max() < synth.TINY.mask_id


# ---- staged token stabilisation (System Design, "Staged Token Stabilization") ----

def _staged_case(rng, n, ties=False):
    conf = rng.random(n).astype(np.float32)
    if ties:
        conf = np.round(conf * 4).astype(np.float32) / 4
    state = rng.integers(0, 3, n).astype(np.uint8)
    mask = (state == oracle.IV).astype(np.uint8)
    pred = rng.integers(0, 1000, n).astype(np.int32)
    tok = np.where(mask == 1, 999, rng.integers(0, 1000, n)).astype(np.int32)
    same = (mask == 0) & (rng.random(n) < 0.5)          # visible rows whose prediction is the held id
    tok[same] = pred[same]
    return conf, pred, tok, mask, state


@pytest.mark.parametrize("seed", range(40))
def test_commit_staged_postconditions(seed):
    """Promoted set, state transitions and untouched positions, from set algebra."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    conf, pred, tok, mask, state = _staged_case(rng, n, ties=bool(seed % 2))
    b = int(rng.integers(0, n))
    ln = int(rng.integers(1, n - b + 1))
    tv, ts = float(rng.choice([0.0, 0.3, 0.5, 0.7, 1.5])), float(rng.choice([0.2, 0.6, 0.9, 2.0]))
    tok0, mask0, state0 = tok.copy(), mask.copy(), state.copy()
    got = oracle.commit_staged(conf, pred, tok, mask, state, b, ln, tv, ts)
    seg = np.zeros(n, bool)
    seg[b:b + ln] = True
    iv = seg & (state0 == oracle.IV)
    above = iv & (conf >= np.float32(tv))
    if above.any():
        want = set(np.flatnonzero(above))
    elif iv.any():
        idx = np.flatnonzero(iv)
        best = idx[conf[idx] == conf[idx].max()].min()      # highest conf, then lowest position
        want = {int(best)}
    else:
        want = set()
    assert set(got.tolist()) == want and list(got) == sorted(got)
    prom = np.zeros(n, bool)
    prom[list(want)] = True
    assert np.array_equal(tok, np.where(prom, pred, tok0))
    assert np.array_equal(mask, np.where(prom, 0, mask0))
    vis_after = prom | (state0 == oracle.V)
    holds = tok == pred                                         # the step predicts the held id
    want_state = np.where(seg & vis_after & holds & (conf >= np.float32(ts)), oracle.S,
                          np.where(prom, oracle.V, state0))
    assert np.array_equal(state, want_state.astype(np.uint8))
    assert np.all(state >= state0)                             # states only move forward


def test_commit_staged_stability_is_a_property_of_the_held_token():
    """A visible token becomes stable only if the step predicts that token: a row that
    now predicts another id at 0.95 keeps its token and stays visible (tracked for
    revision); the same confidence on the held id makes it stable, and a position
    promoted in this step holds its prediction by construction."""
    conf = np.array([0.95, 0.95, 0.95, 0.10], np.float32)
    pred = np.array([5, 6, 7, 8], np.int32)
    tok = np.array([4, 6, 99, 99], np.int32)                # row 0 holds 4 but predicts 5
    mask = np.array([0, 0, 1, 1], np.uint8)
    state = np.array([oracle.V, oracle.V, oracle.IV, oracle.IV], np.uint8)
    got = oracle.commit_staged(conf, pred, tok, mask, state, 0, 4, 0.7, 0.9)
    assert got.tolist() == [2]
    assert state.tolist() == [oracle.V, oracle.S, oracle.S, oracle.IV]
    assert tok.tolist() == [4, 6, 7, 99] and mask.tolist() == [0, 0, 0, 1]


def test_commit_staged_high_threshold_is_top1_commit():
    """theta_visible above every probability: one promotion per step, exactly the k=1 commit."""
    rng = np.random.default_rng(7)
    for _ in range(20):
        n = 24
        conf = (rng.integers(0, 6, n) / 8).astype(np.float32)     # many ties
        pred = rng.integers(0, 50, n).astype(np.int32)
        mask = (rng.random(n) < 0.6).astype(np.uint8)
        state = np.where(mask == 1, oracle.IV, oracle.V).astype(np.uint8)
        tok = np.where(mask == 1, 99, 5).astype(np.int32)
        t2, m2 = tok.copy(), mask.copy()
        got = oracle.commit_staged(conf, pred, tok, mask, state, 0, n, 1.5, 2.0)
        ref = oracle.commit(conf, pred, t2, m2, 0, n, 1)
        assert list(got) == list(ref) and np.array_equal(tok, t2) and np.array_equal(mask, m2)


def test_commit_staged_zero_threshold_reveals_all():
    n = 16
    conf = np.linspace(0.01, 0.99, n).astype(np.float32)
    pred = np.arange(n, dtype=np.int32) + 100
    tok, mask = np.full(n, 7, np.int32), np.ones(n, np.uint8)
    state = np.zeros(n, np.uint8)
    got = oracle.commit_staged(conf, pred, tok, mask, state, 0, n, 0.0, 0.9)
    assert list(got) == list(range(n)) and not mask.any() and np.array_equal(tok, pred)
    assert np.array_equal(state, np.where(conf >= np.float32(0.9), oracle.S, oracle.V))


def test_commit_staged_progress_and_stability():
    """Every step promotes at least one invisible position, so a block of n finishes in
    at most n steps; stable positions never change again."""
    rng = np.random.default_rng(3)
    n = 32
    tok, mask, state = np.full(n, 1023, np.int32), np.ones(n, np.uint8), np.zeros(n, np.uint8)
    for step in range(n):
        conf = rng.random(n).astype(np.float32) ** 4
        pred = rng.integers(0, 1000, n).astype(np.int32)
        before_s = state == oracle.S
        tok_s = tok.copy()
        got = oracle.commit_staged(conf, pred, tok, mask, state, 0, n, 0.7, 0.9)
        assert len(got) >= 1 or not (state == oracle.IV).any()
        assert np.array_equal(tok[before_s], tok_s[before_s]) and np.all(state[before_s] == oracle.S)
        if not mask.any():
            break
    assert not mask.any() and np.all(state != oracle.IV)


# ---- re-prediction of tracked visible prefix tokens ----

STS_SHAPE = dataclasses.replace(MICRO, block=4)


def _sts_prefix(seed=5, P0=8, nb=3):
    """Oracle model, a cache with a prompt and nb appended blocks of random ids, and
    the whole id sequence."""
    sh = STS_SHAPE
    m, _ = micro_model(sh, seed=seed)
    rng = np.random.default_rng(seed)
    seq = rng.integers(0, sh.mask_id, P0 + nb * sh.block).astype(np.int32)
    kv = oracle.OracleKV(sh, len(seq))
    oracle.prefill(m, kv, seq[:P0])
    for b in range(nb):
        oracle.append_block(m, kv, seq[P0 + b * sh.block:P0 + (b + 1) * sh.block])
    return m, kv, seq, P0


def _brute_conf(m, seq, P0, masked):
    """(id, conf) of every position from one full block-causal forward of seq with the
    given positions set to MASK, plus that forward's K/V."""
    s = seq.copy()
    s[list(masked)] = m.shape.mask_id
    allowed = oracle.block_causal_allowed(len(s), P0, m.shape.block)
    _, logits, K, V = oracle.forward_full(m, s, allowed)
    ids, conf = oracle.confidence(logits)
    return ids, conf, K, V


def test_repredict_trailing_blocks_equals_sequential_brute_force():
    """When the tracked set is every position of the last blocks, each block's
    re-prediction sees only fresh K/V, so it equals a full recompute: block b's (id,
    conf) are those of a full block-causal forward with the earlier tracked blocks at
    their new ids and block b hidden (MASK), and the cache afterwards equals a full
    recompute of the final sequence.  A variant that masks more than one block at a
    time (chunks of a fixed row count) or that re-predicts a block before the previous
    one is written back fails this."""
    m, kv, seq, P0 = _sts_prefix()
    B = m.shape.block
    blocks = [list(range(P0 + b * B, P0 + (b + 1) * B)) for b in (1, 2)]
    tracked = {p: int(seq[p]) for blk in blocks for p in blk}
    ids1, conf1, _, _ = _brute_conf(m, seq, P0, blocks[0])
    c = np.sort(conf1[blocks[0]].astype(np.float32))
    tv, ts = float((c[0] + c[1]) / 2), float((c[2] + c[3]) / 2)   # between observed values: no ties
    stable, chosen = oracle.repredict_tracked(m, kv, dict(tracked), tv, ts)
    want, cur, want_stable = {}, seq.copy(), []
    for blk in blocks:
        ids, conf, _, _ = _brute_conf(m, cur, P0, blk)
        for p in blk:
            cf = np.float32(conf[p])
            want[p] = int(ids[p]) if cf >= np.float32(tv) else int(cur[p])
            if cf >= np.float32(ts):
                want_stable.append(p)
        for p in blk:
            cur[p] = want[p]
    assert chosen == want and stable == sorted(want_stable)
    assert 0 < len(stable) < 2 * B and any(want[p] != seq[p] for p in want)    # every branch taken
    _, _, K, V = _brute_conf(m, cur, P0, [])
    np.testing.assert_allclose(kv.K[:, :len(seq)], K, atol=1e-10, rtol=0)
    np.testing.assert_allclose(kv.V[:, :len(seq)], V, atol=1e-10, rtol=0)


def test_repredict_updates_tracking_and_touches_only_tracked_rows():
    """Stable positions leave the tracked set; the others keep the id written back;
    cache rows of untracked positions are unchanged; the thresholds split the
    decisions exactly as stated (conf >= theta_stable -> new id and stable,
    conf >= theta_visible -> new id, otherwise the held id)."""
    m, kv, seq, P0 = _sts_prefix(seed=9, nb=3)
    B = m.shape.block
    tracked = {P0 + 1: int(seq[P0 + 1]), P0 + 3: int(seq[P0 + 3]), P0 + B + 2: int(seq[P0 + B + 2]),
               P0 + 2 * B: int(seq[P0 + 2 * B]), P0 + 2 * B + 3: int(seq[P0 + 2 * B + 3])}
    K0, V0 = kv.K.copy(), kv.V.copy()
    # every position stays: thresholds above 1 keep every held id
    t = dict(tracked)
    stable, chosen = oracle.repredict_tracked(m, kv.copy(), t, 2.0, 3.0)
    assert stable == [] and chosen == tracked and t == tracked
    # theta_visible 0: every position takes its re-predicted id; theta_stable 0: all stable
    t = dict(tracked)
    kv2 = kv.copy()
    stable, chosen = oracle.repredict_tracked(m, kv2, t, 0.0, 0.0)
    assert stable == sorted(tracked) and t == {} and set(chosen) == set(tracked)
    assert all(c != m.shape.mask_id for c in chosen.values())
    untracked = [p for p in range(len(seq)) if p not in tracked]
    np.testing.assert_array_equal(kv2.K[:, untracked], K0[:, untracked])
    np.testing.assert_array_equal(kv2.V[:, untracked], V0[:, untracked])


def test_refresh_of_a_block_and_the_next_block_equals_two_refreshes():
    """The sparse refresh lets two consecutive blocks share one call: rows of block b
    see keys only up to the end of block b, so refreshing block b's rows together with
    block b + 1's rows gives block b's rows the results of a refresh of block b alone,
    and block b + 1's rows those of a second refresh made after it.  (The GPU driver
    merges the write-back of one block with the re-prediction of the next this way.)"""
    m, kv, seq, P0 = _sts_prefix(seed=4, nb=3)
    B, mask_id = m.shape.block, m.shape.mask_id
    wb_pos, wb_ids = [P0 + B + 1, P0 + B + 2], [3, 17]
    mk_pos = [P0 + 2 * B, P0 + 2 * B + 2, P0 + 2 * B + 3]
    kv_a, kv_b = kv.copy(), kv.copy()
    ia, ca, _ = oracle.refresh(m, kv_a, wb_pos + mk_pos, wb_ids + [mask_id] * 3)
    ib1, cb1, _ = oracle.refresh(m, kv_b, wb_pos, wb_ids)
    ib2, cb2, _ = oracle.refresh(m, kv_b, mk_pos, [mask_id] * 3)
    np.testing.assert_array_equal(ia, np.concatenate([ib1, ib2]))
    np.testing.assert_allclose(ca, np.concatenate([cb1, cb2]), rtol=1e-12)
    np.testing.assert_allclose(kv_a.K, kv_b.K, atol=1e-12, rtol=0)
    np.testing.assert_allclose(kv_a.V, kv_b.V, atol=1e-12, rtol=0)
