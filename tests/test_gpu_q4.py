"""Q4_0 weights on the GPU, through the C ABI, against the float64 oracle.

The converter (dllm_quantize_q4_0) must reproduce the oracle's Q4_0 codes and fp16
scales bit for bit: both take every decision in fp32 (the block's signed maximum,
d = m / -8, inv = 1 / d, trunc(x * inv + 8.5) clamped at 15).  The model path
quantises the same way at creation and multiplies with the weights (q - 8) * d
without rounding them, so logits stay within the bf16-activation tolerance of the
oracle's model with dequantised Q4_0 weights.  Small shapes cover ragged K (688:
a half block) and ragged row tiles (vocab 1000), grouped K/V heads with biases, and
the 32 / 48 / 64-row windows; the 8B-width cases sit in test_gpu_8b.
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


def _quantize_gpu(w):
    rows, K = w.shape
    nb = (K + 31) // 32
    if w.dtype == np.uint16:
        src, code = torch.from_numpy(w.view(np.int16)).cuda(), dl.DLLM_BF16
    else:
        src, code = torch.from_numpy(np.ascontiguousarray(w, np.float32)).cuda(), dl.DLLM_F32
    q = torch.full((rows, nb * 32), 0xEE, dtype=torch.uint8, device="cuda")
    d = torch.zeros((rows, nb), dtype=torch.int16, device="cuda")
    dl.dllm_quantize_q4_0(src, code, rows, K, q, d)
    torch.cuda.synchronize()
    return q.cpu().numpy(), d.cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("K", [32, 70, 688, 4096])
@pytest.mark.parametrize("src", ["f32", "bf16"])
def test_quantizer_bit_exact(K, src):
    rng = np.random.default_rng(K)
    rows = 64
    w = (rng.standard_normal((rows, K)) * 0.02).astype(np.float32)
    w[0, :32] = 0.0                                     # an all-zero block
    w[1, 3], w[1, 17] = 0.04, -0.04                     # a sign tie inside one block
    w[2, :32] = np.float32(2.0 ** -7) * (np.arange(32) % 16 - 8)   # a representable block
    w[5] *= 1e-30                                       # tiny values (subnormal fp16 scales)
    if src == "bf16":
        w = synth.normal(K, 3, rows * K, "bf16").reshape(rows, K)
        w[0, :32] = 0
    q, d = _quantize_gpu(w)
    ref_q, ref_d = oracle.quantize_rows_q4_0(synth.as_f32(w))
    np.testing.assert_array_equal(q, ref_q)
    np.testing.assert_array_equal(d, ref_d.view(np.uint16))


def test_quantizer_validation():
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_quantize_q4_0(None, dl.DLLM_F32, 4, 32, None, None)
    assert e.value.code == dl.DLLM_E_INVAL
    buf = torch.zeros(64, device="cuda")
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_quantize_q4_0(buf, dl.DLLM_W8, 1, 32, buf, buf)
    assert e.value.code == dl.DLLM_E_DTYPE


@pytest.fixture(scope="module", params=["small", "tiny_gqa"])
def q4pair(request):
    sh = synth.SMALL_BF16 if request.param == "small" else synth.TINY_GQA
    model, om, _ = build_pair(sh, "q4", max_window=64, max_pos=1024)
    yield sh, model, om
    model.close()


@pytest.mark.parametrize("W", [32, 48, 64])
def test_q4_step_matches_oracle(q4pair, W):
    sh, model, om = q4pair
    print(f"case: Q4_0 d {sh.d_model} heads {sh.n_heads}/{sh.kv_heads} window {W}", flush=True)
    P0 = 100
    kv = dl.KVCache(model, P0 + W)
    okv = oracle.OracleKV(sh, P0 + W)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    oracle.prefill(om, okv, prompt)
    tok, mask = synth.window(sh, W, range(W // 4, W))
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, tol("q4"))
    assert_ids_match_where_decided(ids, ref.logits, err)
    np.testing.assert_allclose(conf, ref.conf, rtol=0.1)
    s_ids, _ = gpu_step(model, kv, tok, mask)
    np.testing.assert_array_equal(s_ids, ids)
    kv.close()


def test_q4_cache_equals_block_causal_recompute(q4pair):
    sh, model, om = q4pair
    print(f"case: Q4_0 cache d {sh.d_model}", flush=True)
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
    Kg, Vt = kv.views()
    n = len(seq)
    np.testing.assert_allclose(Kg[:, :, :n].cpu().numpy(), np.transpose(K, (0, 2, 1, 3)), atol=3e-2, rtol=3e-2)
    np.testing.assert_allclose(Vt[:, :, :, :n].cpu().numpy(), np.transpose(V, (0, 2, 3, 1)), atol=3e-2, rtol=3e-2)
    kv.close()
