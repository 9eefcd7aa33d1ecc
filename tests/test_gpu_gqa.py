"""Grouped-query attention (fewer K/V heads than query heads) and Q/K/V biases on
the GPU, through the C ABI, against the float64 oracle: the Dream-7B model of the
paper's cross-model study.

Small shapes: 4 query heads over 2 K/V heads (fp32 and bf16, head_dim 64) and over
one K/V head (multi-query; bf16 and int8 weights, head_dim 128, ragged FFN and vocab
tiles).  The cache written by prefill and appends is checked against the oracle's
block-causal full recompute, the sparse refresh against the oracle's refresh, and
the Dream-7B widths (d 3584, 28 heads over 4 K/V heads, FFN 18944, vocab 152064) in
the launch configuration the benchmark times.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import (assert_ids_match_where_decided, assert_logits_close, build_pair, dev_i32, gpu_logits,
                      gpu_step, tol)

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402

CASES = [(synth.TINY_GQA, "f32"), (synth.TINY_GQA, "bf16"), (synth.SMALL_MQA, "bf16"), (synth.SMALL_MQA, "w8")]
IDS = ["gqa2-f32", "gqa2-bf16", "mqa-bf16", "mqa-w8"]


@pytest.fixture(scope="module", params=list(range(len(CASES))), ids=IDS)
def pair(request):
    sh, dtype = CASES[request.param]
    model, om, _ = build_pair(sh, dtype, max_window=64, max_pos=1024)
    yield sh, dtype, model, om
    model.close()


def _cache_vs(kv, K_ref, V_ref, n, atol, rtol):
    K, Vt = kv.views()
    Kg = K[:, :, :n].float().cpu().numpy()                      # [L, Hkv, n, Dh]
    Vg = Vt[:, :, :, :n].float().cpu().numpy()                  # [L, Hkv, Dh, n]
    np.testing.assert_allclose(Kg, np.transpose(K_ref[:, :n], (0, 2, 1, 3)), atol=atol, rtol=rtol)
    np.testing.assert_allclose(Vg, np.transpose(V_ref[:, :n], (0, 2, 3, 1)), atol=atol, rtol=rtol)


@pytest.mark.parametrize("W", [32, 48])
def test_gqa_step_matches_oracle(pair, W):
    sh, dtype, model, om = pair
    print(f"case: {sh.n_heads}q/{sh.kv_heads}kv heads {dtype}, prefix 64, window {W}", flush=True)
    P0 = 64
    kv = dl.KVCache(model, P0 + W)
    okv = oracle.OracleKV(sh, P0 + W)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    oracle.prefill(om, okv, prompt)
    tok, mask = synth.window(sh, W, range(W // 4, W))
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, tol(dtype))
    assert_ids_match_where_decided(ids, ref.logits, err)
    np.testing.assert_allclose(conf, ref.conf, rtol=1e-3 if dtype == "f32" else 0.1)
    s_ids, s_conf = gpu_step(model, kv, tok, mask)
    np.testing.assert_array_equal(s_ids, ids)
    kv.close()


def test_gqa_cache_equals_block_causal_recompute(pair):
    sh, dtype, model, om = pair
    print(f"case: cache {sh.n_heads}q/{sh.kv_heads}kv {dtype}", flush=True)
    P0 = 40
    kv = dl.KVCache(model, P0 + 2 * sh.block)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    seq = [prompt]
    for b in range(2):
        blk = synth.uniform_ids(60 + b, 1, sh.block, sh.mask_id)
        dl.dllm_append_prefix_kv(model.handle, kv.handle, dev_i32(blk), sh.block)
        seq.append(blk)
    torch.cuda.synchronize()
    seq = np.concatenate(seq)
    _, _, K, V = oracle.forward_full(om, seq, oracle.block_causal_allowed(len(seq), P0, sh.block))
    atol, rtol = (1e-5, 1e-4) if dtype == "f32" else (3e-2, 3e-2)
    _cache_vs(kv, K, V, len(seq), atol, rtol)
    kv.close()


def test_gqa_long_prompt_cache_equals_recompute(pair):
    """A 300-token prompt (320 padded rows: the bf16 models take the LDS-tiled GEMM,
    with a ragged last token tile and ragged row tiles) then one appended block."""
    sh, dtype, model, om = pair
    print(f"case: long prompt cache {sh.n_heads}q/{sh.kv_heads}kv {dtype}", flush=True)
    P0 = 300
    kv = dl.KVCache(model, P0 + sh.block)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    blk = synth.uniform_ids(90, 1, sh.block, sh.mask_id)
    dl.dllm_append_prefix_kv(model.handle, kv.handle, dev_i32(blk), sh.block)
    torch.cuda.synchronize()
    seq = np.concatenate([prompt, blk])
    _, _, K, V = oracle.forward_full(om, seq, oracle.block_causal_allowed(len(seq), P0, sh.block))
    atol, rtol = (1e-5, 1e-4) if dtype == "f32" else (3e-2, 3e-2)
    _cache_vs(kv, K, V, len(seq), atol, rtol)
    kv.close()


def test_gqa_refresh_matches_oracle(pair):
    sh, dtype, model, om = pair
    print(f"case: refresh {sh.n_heads}q/{sh.kv_heads}kv {dtype}", flush=True)
    P0 = 40
    cap = P0 + 2 * sh.block
    kv = dl.KVCache(model, cap)
    okv = oracle.OracleKV(sh, cap)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    oracle.prefill(om, okv, prompt)
    for b in range(2):
        blk = synth.uniform_ids(70 + b, 1, sh.block, sh.mask_id)
        dl.dllm_append_prefix_kv(model.handle, kv.handle, dev_i32(blk), sh.block)
        oracle.append_block(om, okv, blk)
    pos = np.array([P0 + 3, 7, P0 + sh.block + 30, P0 + sh.block], np.int32)
    new = synth.uniform_ids(80, 1, 4, sh.mask_id)
    ids = torch.empty(4, dtype=torch.int32, device="cuda")
    conf = torch.empty(4, device="cuda")
    dl.dllm_refresh_kv(model.handle, kv.handle, dev_i32(pos), dev_i32(new), 4, ids, conf)
    torch.cuda.synchronize()
    r_ids, r_conf, r_logits = oracle.refresh(om, okv, pos, new, lm_head=True)
    atol = 1e-4 if dtype == "f32" else 5e-2
    _cache_vs(kv, okv.K, okv.V, cap, atol, 1e-3 if dtype == "f32" else 5e-2)
    np.testing.assert_allclose(conf.cpu().numpy(), r_conf, rtol=1e-3 if dtype == "f32" else 0.1)
    assert_ids_match_where_decided(ids.cpu().numpy(), r_logits, atol)
    kv.close()


def _dream_run(n_layers, dtype, W):
    sh = synth.DREAM_7B.with_layers(n_layers)
    P = 512
    print(f"case: Dream-7B width {dtype}, {n_layers} layers, prefix {P}, window {W}", flush=True)
    layers = [synth.layer_weights(sh, l, "bf16") for l in range(n_layers)]
    glob = synth.global_weights(sh, "bf16")
    model = dl.Model(sh, dtype, glob, lambda l: layers[l], max_window=64, max_pos=P + W + 64)
    kv = dl.KVCache(model, P + W)
    prompt = synth.prompt_ids(sh, P)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P)
    masked = list(range(8, 32)) if W == 32 else list(range(24, 64))
    tok, mask = synth.window(sh, W, masked)
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    print("  gpu done; oracle ...", flush=True)
    om = oracle.OracleModel(sh, dict(glob, layers=layers), cache_layers=False)
    okv = oracle.OracleKV(sh, P + W)
    oracle.prefill(om, okv, prompt)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, tol(dtype))
    frac = assert_ids_match_where_decided(ids, ref.logits, err)
    print(f"  max |dlogit| = {err:.3e}; argmax decided on {frac:.0%} of rows", flush=True)
    np.testing.assert_allclose(conf, ref.conf, rtol=0.2)
    kv.close()
    model.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("dtype,W", [("bf16", 32), ("bf16", 64)])
def test_dream7b_width_two_layers(dtype, W):
    _dream_run(2, dtype, W)


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_dream7b_full_depth_step():
    """All 28 layers of the Dream-7B shape (grouped-query attention over 4 K/V heads, Q/K/V
    biases), the 32-row window at prefix 512 that its workload times."""
    _dream_run(synth.DREAM_7B.n_layers, "bf16", 32)
