"""Selective logits skipping on the GPU, through the C ABI.

dllm_denoise_window_sls runs the LM head over the selected rows only, packed to the
front.  Checked against the oracle's denoise_window_sls (same seeded inputs,
tolerance of the model's dtype) and against the library's own unselected step: the
kept rows' ids must be identical and their confidences equal to fp32 rounding (the
LM head's per-row arithmetic does not depend on a row's slot; only the split of the
exp-sum over lanes follows the packed row count), the other rows (-1, 0), and the
K/V the step writes bit-identical.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_ids_match_where_decided, build_pair, dev_i32, dev_u8, tol

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402


def _sls(model, kv, w0, tok, mask, need, n_need):
    W = len(tok)
    ids = torch.full((W,), 7, dtype=torch.int32, device="cuda")
    conf = torch.full((W,), 7.0, device="cuda")
    d_need = None if need is None else dev_u8(need)
    dl.dllm_denoise_window_sls(model.handle, kv.handle, w0, dev_i32(tok), dev_u8(mask), d_need, n_need, W, ids,
                               conf)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), conf.cpu().numpy().astype(np.float64)


def _full(model, kv, w0, tok, mask):
    W = len(tok)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    dl.dllm_denoise_window(model.handle, kv.handle, w0, dev_i32(tok), dev_u8(mask), W, ids, conf)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), conf.cpu().numpy().astype(np.float64)


def _kv_copy(kv):
    K, Vt = kv.views()
    return K.clone(), Vt.clone()


def _check_against_full(ids, conf, full_ids, full_conf, need, n_need):
    W = len(ids)
    flag = np.ones(W, bool) if need is None else need != 0
    kept = np.flatnonzero(flag)[:n_need]
    skipped = np.setdiff1d(np.arange(W), kept)
    np.testing.assert_array_equal(ids[kept], full_ids[kept])
    np.testing.assert_allclose(conf[kept], full_conf[kept], rtol=1e-5, atol=0)
    assert np.all(ids[skipped] == -1) and np.all(conf[skipped] == 0.0)
    return kept


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("W", [32, 48, 64])
def test_sls_matches_full_step_and_oracle(dtype, W):
    sh = synth.TINY if dtype == "f32" else synth.SMALL_BF16
    model, om, _ = build_pair(sh, dtype, max_pos=512)
    P0 = 64
    kv = dl.KVCache(model, P0 + W)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    okv = oracle.OracleKV(sh, P0 + W)
    oracle.prefill(om, okv, prompt)
    rng = np.random.default_rng(W)
    masked = sorted(rng.choice(W, (2 * W) // 3, replace=False).tolist())
    tok, mask = synth.window(sh, W, masked)
    full_ids, full_conf = _full(model, kv, P0, tok, mask)
    K0, V0 = _kv_copy(kv)
    n_mask = int(mask.sum())
    cases = [(mask, n_mask), (mask, n_mask - 5), (mask, 0), (mask, W), (None, 17), (None, W)]
    for need, n_need in cases:
        print(f"case: sls {dtype} W {W} n_need {n_need} need {'mask' if need is not None else 'all'}", flush=True)
        ids, conf = _sls(model, kv, P0, tok, mask, need, n_need)
        _check_against_full(ids, conf, full_ids, full_conf, need, n_need)
        K1, V1 = _kv_copy(kv)
        assert torch.equal(K0, K1) and torch.equal(V0, V1)
    # the oracle's selective step on the same inputs
    o_ids, o_conf, so = oracle.denoise_window_sls(om, okv, P0, tok, mask, mask, n_mask - 5)
    ids, conf = _sls(model, kv, P0, tok, mask, mask, n_mask - 5)
    kept = np.flatnonzero(mask)[:n_mask - 5]
    np.testing.assert_array_equal(ids == -1, o_ids == -1)
    np.testing.assert_array_equal(conf == 0.0, o_conf == 0.0)
    np.testing.assert_allclose(conf[kept], o_conf[kept], rtol=1e-3 if dtype == "f32" else 0.1)
    assert_ids_match_where_decided(ids[kept], so.logits[kept], tol(dtype))
    kv.close()
    model.close()


def test_sls_validation():
    sh = synth.TINY
    model, _, _ = build_pair(sh, "f32", max_pos=256, oracle_too=False)
    kv = dl.KVCache(model, 128)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(sh, 32)), 32)
    tok, mask = synth.window(sh, 16, range(16))
    for w0, n_need, W, code in [(32, -1, 16, dl.DLLM_E_INVAL), (32, 17, 16, dl.DLLM_E_INVAL),
                                (31, 4, 16, dl.DLLM_E_INVAL), (120, 4, 16, dl.DLLM_E_CAPACITY)]:
        with pytest.raises(dl.DllmError) as e:
            _sls(model, kv, w0, tok[:W], mask[:W], None, n_need)
        assert e.value.code == code
    kv.close()
    model.close()


@pytest.mark.timeout(600)
def test_sls_8b_width_spec_window():
    """The speculative 64-row window at the LLaDA-8B widths (2 layers): 40 masked
    rows run the LM head at 48 packed rows instead of 64; the kept rows equal the
    unselected step's (which the 8B-width parity test checks against the oracle)."""
    sh = synth.LLADA_8B.with_layers(2)
    layers = [synth.layer_weights(sh, l, "bf16") for l in range(2)]
    glob = synth.global_weights(sh, "bf16")
    model = dl.Model(sh, "bf16", glob, lambda l: layers[l], max_window=64, max_pos=1024 + 128)
    P, W = 1024, 64
    kv = dl.KVCache(model, P + W)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(sh, P)), P)
    tok, mask = synth.window(sh, W, list(range(24, 64)))
    print("case: sls 8B width, P 1024, W 64, 40 masked", flush=True)
    full_ids, full_conf = _full(model, kv, P, tok, mask)
    for n_need in (40, 16):
        ids, conf = _sls(model, kv, P, tok, mask, mask, n_need)
        _check_against_full(ids, conf, full_ids, full_conf, mask, n_need)
    kv.close()
    model.close()
