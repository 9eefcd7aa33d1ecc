"""Full-width parity at the LLaDA-8B shape (d 4096, 32 heads x 128, FFN 12288,
vocab 126464) in the launch configuration the benchmark times.

The kernels' launch shapes depend only on the widths and the window size, so
the 2-layer cases exercise exactly the benchmark's GEMM, attention and LM-head
launches; the full 32-layer case compares one whole step at prefix 512 with
the oracle (it takes about a minute of CPU time on the host).
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_ids_match_where_decided, assert_logits_close, dev_i32, dev_u8, gpu_logits, gpu_step, tol

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402

BIG = synth.LLADA_8B


def _host_gib_available():
    try:
        import psutil
        return psutil.virtual_memory().available / 2**30
    except Exception:
        return 0.0


def _sls_step(model, kv, tok, mask, n_need):
    """The benchmark's speculative-window call: dllm_denoise_window_sls at w0 = P with
    the mask as the need flags (only masked rows get an LM-head output)."""
    W = len(tok)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    d_mask = dev_u8(mask)
    dl.dllm_denoise_window_sls(model.handle, kv.handle, kv.prefix_len, dev_i32(tok), d_mask, d_mask, n_need, W,
                               ids, conf)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), conf.cpu().numpy().astype(np.float64)


def _run(shape, dtype, P, W, masked, cap_extra=0, sls=False):
    print(f"case: 8B-width {dtype}, layers {shape.n_layers}, prefix {P}, window {W}"
          f"{', selective logits' if sls else ''}", flush=True)
    layers = [synth.layer_weights(shape, l, "bf16") for l in range(shape.n_layers)]
    glob = synth.global_weights(shape, "bf16")
    model = dl.Model(shape, dtype, glob, lambda l: layers[l], max_window=64, max_pos=P + W + 64)
    kv = dl.KVCache(model, P + W + cap_extra)
    prompt = synth.prompt_ids(shape, P)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P)
    tok, mask = synth.window(shape, W, masked)
    logits, ids, conf = gpu_logits(model, kv, tok, mask)
    s_ids, s_conf = gpu_step(model, kv, tok, mask)
    if sls:
        l_ids, l_conf = _sls_step(model, kv, tok, mask, len(masked))
        kept = mask != 0
        np.testing.assert_array_equal(l_ids[kept], ids[kept])
        np.testing.assert_allclose(l_conf[kept], conf[kept], rtol=1e-5, atol=0)
        assert np.all(l_ids[~kept] == -1) and np.all(l_conf[~kept] == 0.0)
    print("  gpu done; oracle ...", flush=True)
    # the float64 oracle converts a layer's weights on each use; keep them when the host
    # has room for all of them (the quantised paths convert slowly)
    cache = shape.params_per_layer * shape.n_layers * 8 < (_host_gib_available() - 48) * 2**30
    om = oracle.OracleModel(shape, dict(glob, layers=layers), int8=(dtype == "w8"), q4=(dtype == "q4"),
                            cache_layers=cache)
    okv = oracle.OracleKV(shape, P + W + cap_extra)
    oracle.prefill(om, okv, prompt)
    ref = oracle.denoise_step(om, okv, tok, mask)
    err = assert_logits_close(logits, ref.logits, tol(dtype))
    frac = assert_ids_match_where_decided(ids, ref.logits, err)
    print(f"  max |dlogit| = {err:.3e}; argmax decided on {frac:.0%} of rows", flush=True)
    np.testing.assert_array_equal(s_ids, ids)
    np.testing.assert_array_equal(s_conf, conf)
    np.testing.assert_allclose(conf, ref.conf, rtol=0.2)
    assert np.all(ids != shape.mask_id) and np.all((conf > 0) & (conf <= 1))
    kv.close()
    model.close()
    return err


@pytest.mark.timeout(600)
@pytest.mark.parametrize("dtype,P,W", [("bf16", 512, 32), ("bf16", 512, 48), ("bf16", 1024, 64), ("w8", 512, 64),
                                       ("q4", 512, 32), ("q4", 512, 48), ("q4", 512, 64), ("bf16", 440, 32)])
def test_8b_width_two_layers(dtype, P, W):
    """The bench's launches at the 8B widths; the 440-token prompt (448 rows) takes the
    prompt's split-K QKV with a ragged second token group (12 of 16 token tiles)."""
    masked = list(range(8, 32)) if W == 32 else list(range(24, W))
    _run(BIG.with_layers(2), dtype, P, W, masked)


@pytest.mark.timeout(900)
def test_8b_width_long_prefix_int8_spec_window():
    """The long-prefix int8 speculative launch configuration at the 8B widths: int8
    weights, a 64-row window, and a prefix long enough that the attention's key
    splits hit their cap (2048 keys: 66 blocks in 14 splits; the 4096-key workload
    takes 15 splits through the same code).  One layer: the oracle's prefill is the
    cost."""
    _run(BIG.with_layers(1), "w8", 2048, 64, list(range(0, 64)))


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_8b_full_depth_step():
    _run(BIG, "bf16", 512, 32, list(range(8, 32)))


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_8b_full_depth_q4_step():
    """32 layers of Q4_0 weights (the converter's codes and fp16 block scales), the
    32-row window at prefix 512 that the Q4_0 workload times."""
    _run(BIG, "q4", 512, 32, list(range(8, 32)))


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_8b_full_depth_int8_spec_window_sls():
    """32 layers of int8 weights, a 64-row all-MASK window (current + speculative
    block) through the benchmark's selective-logits call, prefix 512."""
    _run(BIG, "w8", 512, 64, list(range(0, 64)), sls=True)


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_8b_width_int8_prefix_4096_spec_window():
    """The long-prefix int8 workload's launches at its own prefix: 4096 keys + the
    64-row window = 130 key blocks in 15 attention splits, through the selective-logits
    call the benchmark makes.  Two layers (the oracle's 4096-token prefill is the cost)."""
    _run(BIG.with_layers(2), "w8", 4096, 64, list(range(0, 64)), sls=True)


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_8b_full_depth_bf16_spec_window_prefix_1024():
    """32 layers, bf16, prefix 1024, a 64-row window with 8 MASK in the current block
    and an all-MASK speculative block, through the selective-logits call."""
    _run(BIG, "bf16", 1024, 64, list(range(24, 64)), sls=True)


@pytest.mark.timeout(600)
def test_8b_width_append_and_refresh():
    """The end-to-end generation's cache calls at the 8B widths (2 layers): a 512-token
    prefill, two 32-token block appends, then a sparse refresh of 4 revised positions (two
    in the prompt, two in the appended blocks: 4 rows with their own key limits) with
    its LM-head outputs.  The whole cache and the refresh's ids / confidences against the
    oracle."""
    sh = BIG.with_layers(2)
    P0, B = 512, sh.block
    cap = P0 + 2 * B
    print(f"case: 8B-width bf16, 2 layers, prefill {P0}, 2 appends of {B}, refresh of 4 rows", flush=True)
    layers = [synth.layer_weights(sh, l, "bf16") for l in range(sh.n_layers)]
    glob = synth.global_weights(sh, "bf16")
    model = dl.Model(sh, "bf16", glob, lambda l: layers[l], max_window=64, max_pos=cap + 64)
    kv = dl.KVCache(model, cap)
    om = oracle.OracleModel(sh, dict(glob, layers=layers), cache_layers=True)
    okv = oracle.OracleKV(sh, cap)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    oracle.prefill(om, okv, prompt)
    for b in range(2):
        blk = synth.uniform_ids(90 + b, 1, B, sh.mask_id)
        dl.dllm_append_prefix_kv(model.handle, kv.handle, dev_i32(blk), B)
        oracle.append_block(om, okv, blk)
    pos = np.array([P0 + 3, 7, P0 + B + 30, P0 + B], np.int32)
    new = synth.uniform_ids(95, 1, 4, sh.mask_id)
    ids = torch.empty(4, dtype=torch.int32, device="cuda")
    conf = torch.empty(4, device="cuda")
    dl.dllm_refresh_kv(model.handle, kv.handle, dev_i32(pos), dev_i32(new), 4, ids, conf)
    torch.cuda.synchronize()
    assert kv.prefix_len == cap
    r_ids, r_conf, r_logits = oracle.refresh(om, okv, pos, new, lm_head=True)
    K, Vt = kv.views()
    Kg = K[:, :, :cap].float().cpu().numpy()                      # [L, Hkv, n, Dh]
    Vg = Vt[:, :, :, :cap].float().cpu().numpy()                  # [L, Hkv, Dh, n]
    Kr = np.transpose(okv.K[:, :cap], (0, 2, 1, 3))
    Vr = np.transpose(okv.V[:, :cap], (0, 2, 3, 1))
    err = max(float(np.abs(Kg - Kr).max()), float(np.abs(Vg - Vr).max()))
    print(f"  cache max |dK|, |dV| = {err:.3e}", flush=True)
    np.testing.assert_allclose(Kg, Kr, atol=5e-2, rtol=5e-2)
    np.testing.assert_allclose(Vg, Vr, atol=5e-2, rtol=5e-2)
    np.testing.assert_allclose(conf.cpu().numpy(), r_conf, rtol=0.1)
    assert_ids_match_where_decided(ids.cpu().numpy(), r_logits, 5e-2)
    kv.close()
    model.close()
