"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Small shapes that span several tiles and ragged tails: the tiny fp32 model
(d 256, FFN 688, vocab 1024), a micro fp32 model, and a bf16 / int8 model with
head_dim 128, FFN 688 (a ragged K tail in bf16 chunks) and vocab 1000 (a ragged
row tile).  Tolerances: logits 1e-4 (fp32), 5e-2 (bf16, int8 weights).
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import (assert_ids_match_where_decided, assert_logits_close, build_pair, dev_i32, dev_u8,
                      gpu_logits, gpu_step, tol)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402

SMALL = synth.SMALL_BF16


def _prefilled(model, om, shape, P0, cap):
    prompt = synth.prompt_ids(shape, P0)
    kv = dl.KVCache(model, cap)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    okv = oracle.OracleKV(shape, cap)
    oracle.prefill(om, okv, prompt)
    return kv, okv, prompt


@pytest.fixture(scope="module")
def tiny():
    model, om, _ = build_pair(synth.TINY, "f32", max_pos=512)
    yield model, om
    model.close()


@pytest.fixture(scope="module")
def micro():
    model, om, _ = build_pair(synth.MICRO, "f32", max_window=256, max_pos=1024)
    yield model, om
    model.close()


@pytest.fixture(scope="module", params=["bf16", "w8"])
def small(request):
    model, om, _ = build_pair(SMALL, request.param, max_pos=1024)
    yield model, om, request.param
    model.close()


def test_tiny_fp32_step(tiny):
    model, om = tiny
    sh = synth.TINY
    print("case: tiny fp32, prefill 64, window 32 all MASK", flush=True)
    kv, okv, _ = _prefilled(model, om, sh, 64, 96)
    tok, mask = synth.window(sh, 32, range(32))
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, 1e-4)
    assert_ids_match_where_decided(ids, ref.logits, err)
    np.testing.assert_allclose(conf, ref.conf, rtol=1e-3)
    assert np.all(ids != sh.mask_id)
    kv.close()


def test_tiny_generation_with_resync(tiny):
    """4 denoising steps x top-8 commits over a 32-token all-MASK block."""
    model, om = tiny
    sh = synth.TINY
    kv, okv, _ = _prefilled(model, om, sh, 64, 96)
    tok, mask = synth.window(sh, 32, range(32))
    for step, k in enumerate(oracle.commit_schedule(32, 4)):
        print(f"case: tiny generation step {step}", flush=True)
        logits, ids, conf = gpu_logits(model, kv, tok, mask)
        ref = oracle.denoise_step(om, okv, tok, mask)
        err = assert_logits_close(logits, ref.logits, 1e-4)
        assert_ids_match_where_decided(ids, ref.logits, err)
        # the GPU commit on the GPU's own predictions
        t_tok, t_mask = dev_i32(tok), dev_u8(mask)
        cpos = torch.full((k,), -1, dtype=torch.int32, device="cuda")
        ncom = torch.zeros(1, dtype=torch.int32, device="cuda")
        dl.dllm_commit(torch.from_numpy(conf.astype(np.float32)).cuda(), dev_i32(ids), t_tok, t_mask, 0, 32, k,
                       cpos, ncom)
        torch.cuda.synchronize()
        mask_before = mask.copy()
        g_tok, g_mask = tok.copy(), mask.copy()
        ref_pos = oracle.commit(conf, ids, g_tok, g_mask, 0, 32, k)
        assert int(ncom.item()) == min(k, int(mask_before.sum()))
        np.testing.assert_array_equal(cpos.cpu().numpy(), ref_pos)
        np.testing.assert_array_equal(t_tok.cpu().numpy(), g_tok)
        np.testing.assert_array_equal(t_mask.cpu().numpy(), g_mask)
        # resync: continue from the oracle's own commit
        oracle.commit(ref.conf, ref.ids, tok, mask, 0, 32, k)
    assert mask.sum() == 0
    kv.close()


@pytest.mark.parametrize("W", [1, 5, 16, 31, 33, 40, 48, 49, 64, 100, 256])
def test_micro_window_sizes(micro, W):
    model, om = micro
    sh = synth.MICRO
    print(f"case: micro fp32 window {W}", flush=True)
    kv, okv, _ = _prefilled(model, om, sh, 37, 37 + W)
    tok, mask = synth.window(sh, W, range(0, W, 2))
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, 1e-4)
    assert_ids_match_where_decided(ids, ref.logits, err)
    kv.close()


@pytest.mark.parametrize("W", [32, 44, 48, 64])
def test_small_lowp_step(small, W):
    model, om, dtype = small
    sh = SMALL
    print(f"case: small {dtype} window {W}", flush=True)
    kv, okv, _ = _prefilled(model, om, sh, 100, 100 + W)
    tok, mask = synth.window(sh, W, range(W // 4, W))
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, tol(dtype))
    print(f"  max |dlogit| = {err:.3e}", flush=True)
    assert_ids_match_where_decided(ids, ref.logits, err)
    np.testing.assert_allclose(conf, ref.conf, rtol=0.1)
    kv.close()


def test_small_bf16_max_window_and_long_prefill():
    """The largest window a model allows (max_window = 256: four 64-row token blocks
    per launch) and a 1000-token prompt (16 token blocks, ragged), bf16."""
    sh = SMALL
    model, om, _ = build_pair(sh, "bf16", max_window=256, max_pos=1400)
    P0, W = 1000, 256
    print(f"case: small bf16 prefill {P0}, window {W}", flush=True)
    kv, okv, prompt = _prefilled(model, om, sh, P0, P0 + W)
    allowed = oracle.block_causal_allowed(P0, P0, sh.block)
    _, _, K, V = oracle.forward_full(om, prompt, allowed)
    _cache_vs(kv, K, V, P0, 3e-2, 3e-2)
    tok, mask = synth.window(sh, W, range(0, W, 3))
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, tol("bf16"))
    assert_ids_match_where_decided(ids, ref.logits, err)
    kv.close()
    model.close()


def _cache_vs(kv, K_ref, V_ref, n, atol, rtol):
    K, Vt = kv.views()
    Kg = K[:, :, :n].float().cpu().numpy()                      # [L, H, n, Dh]
    Vg = Vt[:, :, :, :n].float().cpu().numpy()                  # [L, H, Dh, n]
    Kr = np.transpose(K_ref[:, :n], (0, 2, 1, 3))
    Vr = np.transpose(V_ref[:, :n], (0, 2, 3, 1))
    np.testing.assert_allclose(Kg, Kr, atol=atol, rtol=rtol)
    np.testing.assert_allclose(Vg, Vr, atol=atol, rtol=rtol)


@pytest.mark.parametrize("which", ["micro", "small_bf16"])
def test_prefill_append_cache_equals_bruteforce(which, micro):
    """GPU cache after prefill + 2 appends = K/V of one block-causal full forward."""
    if which == "micro":
        model, om = micro
        sh, atol, rtol = synth.MICRO, 2e-5, 1e-4
    else:
        model, om, _ = build_pair(SMALL, "bf16", max_pos=1024)
        sh, atol, rtol = SMALL, 3e-2, 3e-2
    print(f"case: cache brute force {which}", flush=True)
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
    assert kv.prefix_len == len(seq)
    _, _, K, V = oracle.forward_full(om, seq, oracle.block_causal_allowed(len(seq), P0, sh.block))
    _cache_vs(kv, K, V, len(seq), atol, rtol)
    kv.close()
    if which != "micro":
        model.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_refresh_matches_oracle(dtype, micro):
    if dtype == "f32":
        model, om = micro
        sh, atol = synth.MICRO, 1e-4
    else:
        model, om, _ = build_pair(SMALL, "bf16", max_pos=1024)
        sh, atol = SMALL, 5e-2
    print(f"case: refresh {dtype}", flush=True)
    P0 = 40
    cap = P0 + 2 * sh.block
    kv, okv, _ = _prefilled(model, om, sh, P0, cap)
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
    _cache_vs(kv, okv.K, okv.V, cap, atol, 1e-3 if dtype == "f32" else 5e-2)
    np.testing.assert_allclose(conf.cpu().numpy(), r_conf, rtol=1e-3 if dtype == "f32" else 0.1)
    assert_ids_match_where_decided(ids.cpu().numpy(), r_logits, atol)
    kv.close()
    if dtype != "f32":
        model.close()


def test_commit_kernel_bit_exact():
    rng = np.random.default_rng(11)
    for trial in range(60):
        n = int(rng.integers(1, 300))
        conf = rng.choice(np.float32([0.1, 0.2, 0.25, 0.5, 0.7]), size=n).astype(np.float32)
        if trial % 3 == 0:
            conf = rng.random(n).astype(np.float32)
        mask = rng.integers(0, 2, size=n).astype(np.uint8)
        pred = rng.integers(0, 1000, size=n).astype(np.int32)
        tok = rng.integers(0, 1000, size=n).astype(np.int32)
        b = int(rng.integers(0, n))
        ln = int(rng.integers(0, n - b + 1))
        k = int(rng.integers(0, 12))
        t_tok, t_mask = dev_i32(tok), dev_u8(mask)
        cpos = torch.full((max(k, 1),), -1, dtype=torch.int32, device="cuda")
        ncom = torch.zeros(1, dtype=torch.int32, device="cuda")
        dl.dllm_commit(torch.from_numpy(conf).cuda(), dev_i32(pred), t_tok, t_mask, b, ln, k, cpos, ncom)
        torch.cuda.synchronize()
        m0 = mask.copy()
        ref = oracle.commit(conf, pred, tok, mask, b, ln, k)
        assert int(ncom.item()) == len(ref) == min(k, int(m0[b:b + ln].sum()))
        np.testing.assert_array_equal(cpos.cpu().numpy()[:len(ref)], ref)
        np.testing.assert_array_equal(t_tok.cpu().numpy(), tok)
        np.testing.assert_array_equal(t_mask.cpu().numpy(), mask)


def test_step_is_deterministic_and_matches_debug(small):
    model, om, dtype = small
    sh = SMALL
    kv, _, _ = _prefilled(model, om, sh, 64, 128)
    tok, mask = synth.window(sh, 64, range(8, 64))
    a_ids, a_conf = gpu_step(model, kv, tok, mask)
    b_ids, b_conf = gpu_step(model, kv, tok, mask)
    np.testing.assert_array_equal(a_ids, b_ids)
    np.testing.assert_array_equal(a_conf, b_conf)
    l1, d_ids, d_conf = gpu_logits(model, kv, tok, mask)
    l2, _, _ = gpu_logits(model, kv, tok, mask)
    np.testing.assert_array_equal(l1, l2)
    np.testing.assert_array_equal(a_ids, d_ids)
    np.testing.assert_array_equal(a_conf, d_conf)
    kv.close()


def test_kernel_replay_leaves_the_prefix_and_later_steps_unchanged(small):
    """dllm_kernel_replay (timing) relaunches the step's kernels on workspace and
    window scratch only: the prefix cache stays bit-identical and the next step
    gives bit-identical outputs."""
    model, om, dtype = small
    sh = SMALL
    kv, okv, _ = _prefilled(model, om, sh, 70, 70 + 32)
    tok, mask = synth.window(sh, 32, range(8, 32))
    ids0, conf0 = gpu_step(model, kv, tok, mask)
    K0, V0 = kv.views()
    for cls in range(6):
        dl.dllm_kernel_replay(model.handle, kv.handle, cls, 32, 5)
    torch.cuda.synchronize()
    K1, V1 = kv.views()
    assert torch.equal(K0[:, :, :70], K1[:, :, :70]) and torch.equal(V0[:, :, :, :70], V1[:, :, :, :70])
    ids1, conf1 = gpu_step(model, kv, tok, mask)
    np.testing.assert_array_equal(ids0, ids1)
    np.testing.assert_array_equal(conf0, conf1)
    with pytest.raises(dl.DllmError):
        dl.dllm_kernel_replay(model.handle, kv.handle, 6, 32, 1)
    kv.close()


def test_window_never_touches_prefix(small):
    """A step (drafts included) leaves cache rows [0, P) and prefix_len unchanged."""
    model, om, dtype = small
    sh = SMALL
    kv, _, _ = _prefilled(model, om, sh, 64, 128)
    K, Vt = kv.views()
    K0, V0 = K[:, :, :64].clone(), Vt[:, :, :, :64].clone()
    gpu_step(model, kv, *synth.window(sh, 64, range(64)))
    assert kv.prefix_len == 64
    assert torch.equal(K[:, :, :64], K0) and torch.equal(Vt[:, :, :, :64], V0)
    kv.close()


def test_host_validation_errors(micro):
    model, _ = micro
    kv = dl.KVCache(model, 64)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(np.arange(40)), 40)
    tok = dev_i32(np.zeros(32))
    out_i = torch.empty(32, dtype=torch.int32, device="cuda")
    out_c = torch.empty(32, device="cuda")
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_denoise_step(model.handle, kv.handle, tok, None, 32, out_i, out_c)   # 40 + 32 > 64
    assert e.value.code == dl.DLLM_E_CAPACITY
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_refresh_kv(model.handle, kv.handle, dev_i32([3, 3]), dev_i32([1, 2]), 2)
    assert e.value.code == dl.DLLM_E_INVAL
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_refresh_kv(model.handle, kv.handle, dev_i32([45]), dev_i32([1]), 1)
    assert e.value.code == dl.DLLM_E_INVAL
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_prefill(model.handle, kv.handle, tok, 8)
    assert e.value.code == dl.DLLM_E_INVAL
    assert kv.prefix_len == 40
    kv.close()
