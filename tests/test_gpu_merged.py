"""Piggybacked append and refresh (dllm_step_merged) against the oracle.

One GPU forward over [refresh rows | completed block | window] must equal, row for
row, the oracle's sequence refresh -> append -> denoising step (the delayed merge
of revisions and the completed block, System Design).  Each group alone must
equal the single-purpose entry point on the GPU.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_ids_match_where_decided, build_pair, dev_i32, dev_u8

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402


def _cache(kv, n):
    K, Vt = kv.views()
    return K[:, :, :n].float().cpu().numpy(), np.swapaxes(Vt[:, :, :, :n].float().cpu().numpy(), 2, 3)


def _oracle_cache(okv, n):
    return np.transpose(okv.K[:, :n], (0, 2, 1, 3)), np.transpose(okv.V[:, :n], (0, 2, 1, 3))


def _merged(model, kv, ref_pos, ref_new, blk, tok, mask):
    n_ref, n_blk, W = len(ref_pos), len(blk), len(tok)
    out = [torch.empty(W, dtype=torch.int32, device="cuda"), torch.empty(W, device="cuda")]
    rout = [torch.empty(max(n_ref, 1), dtype=torch.int32, device="cuda"), torch.empty(max(n_ref, 1), device="cuda")]
    dl.dllm_step_merged(model.handle, kv.handle, dev_i32(ref_pos) if n_ref else None,
                        dev_i32(ref_new) if n_ref else None, n_ref, dev_i32(blk) if n_blk else None, n_blk,
                        dev_i32(tok) if W else None, dev_u8(mask) if W else None, W,
                        out[0] if W else None, out[1] if W else None,
                        rout[0] if n_ref else None, rout[1] if n_ref else None)
    torch.cuda.synchronize()
    return (out[0].cpu().numpy(), out[1].cpu().numpy().astype(np.float64),
            rout[0].cpu().numpy()[:n_ref], rout[1].cpu().numpy()[:n_ref].astype(np.float64))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", ["f32", "bf16", "bf16_8b_width"])
def test_merged_matches_sequential_oracle(case):
    """Small shapes, and the 8B widths (2 layers) near the merged generation's configuration:
    a 512-token prompt, 4 refresh rows + a 32-token block + a 28-row window (64 rows, the
    models' window limit)."""
    dtype = "f32" if case == "f32" else "bf16"
    sh = {"f32": synth.MICRO, "bf16": synth.SMALL_BF16, "bf16_8b_width": synth.LLADA_8B.with_layers(2)}[case]
    atol, crtol = (1e-4, 1e-3) if dtype == "f32" else (5e-2, 0.1)
    B, P0, W = (sh.block, 512, 28) if case == "bf16_8b_width" else (sh.block, 40, 20)
    cap = P0 + 3 * B + W
    model, om, _ = build_pair(sh, dtype, max_pos=max(512, cap + 64))
    kv = dl.KVCache(model, cap)
    okv = oracle.OracleKV(sh, cap)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    oracle.prefill(om, okv, prompt)
    blk1 = synth.uniform_ids(70, 1, B, sh.mask_id)
    dl.dllm_append_prefix_kv(model.handle, kv.handle, dev_i32(blk1), B)
    oracle.append_block(om, okv, blk1)
    P = P0 + B
    ref_pos = np.array([5, P0 + 3, P - 1, 17], np.int32)         # prompt and the earlier block
    ref_new = synth.uniform_ids(81, 1, 4, sh.mask_id)
    blk2 = synth.uniform_ids(71, 1, B, sh.mask_id)
    tok, mask = synth.window(sh, W, range(4, W))
    print(f"case: merged {case}: 4 refresh + {B} append + {W} window rows at prefix {P}", flush=True)
    ids, conf, rids, rconf = _merged(model, kv, ref_pos, ref_new, blk2, tok, mask)
    r_ids, r_conf, r_logits = oracle.refresh(om, okv, ref_pos, ref_new, lm_head=True)
    oracle.append_block(om, okv, blk2)
    so = oracle.denoise_step(om, okv, tok, mask)
    assert kv.prefix_len == P + B == okv.prefix_len
    n = P + B + W
    (Kg, Vg), (Kr, Vr) = _cache(kv, n), _oracle_cache(okv, n)
    np.testing.assert_allclose(Kg, Kr, atol=atol, rtol=crtol)
    np.testing.assert_allclose(Vg, Vr, atol=atol, rtol=crtol)
    np.testing.assert_allclose(conf, so.conf, rtol=crtol)
    np.testing.assert_allclose(rconf, r_conf, rtol=crtol)
    assert_ids_match_where_decided(ids, so.logits, atol)
    assert_ids_match_where_decided(rids, r_logits, atol)
    # the next step sees the merged prefix: same result as the oracle's
    tok2, mask2 = synth.window(sh, W, range(W), seed=5)
    out_i = torch.empty(W, dtype=torch.int32, device="cuda")
    out_c = torch.empty(W, device="cuda")
    dl.dllm_denoise_step(model.handle, kv.handle, dev_i32(tok2), dev_u8(mask2), W, out_i, out_c)
    torch.cuda.synchronize()
    so2 = oracle.denoise_step(om, okv, tok2, mask2)
    np.testing.assert_allclose(out_c.cpu().numpy(), so2.conf, rtol=crtol)
    kv.close()
    model.close()


def test_merged_single_groups_equal_the_single_calls():
    """Each group alone through dllm_step_merged equals the dedicated entry point (fp32 model)."""
    sh = synth.TINY
    model, _, _ = build_pair(sh, "f32", max_pos=512, oracle_too=False)
    B, P0, W = sh.block, 64, 24
    cap = P0 + 2 * B + W

    def fresh():
        kv = dl.KVCache(model, cap)
        dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(sh, P0)), P0)
        return kv

    blk = synth.uniform_ids(72, 1, B, sh.mask_id)
    tok, mask = synth.window(sh, W, range(0, W, 2))
    ref_pos = np.array([3, 60, 11], np.int32)
    ref_new = synth.uniform_ids(82, 1, 3, sh.mask_id)
    print("case: merged single groups (tiny fp32)", flush=True)
    # window only == denoise step
    a, b = fresh(), fresh()
    ids, conf, _, _ = _merged(model, a, [], [], [], tok, mask)
    out_i = torch.empty(W, dtype=torch.int32, device="cuda")
    out_c = torch.empty(W, device="cuda")
    dl.dllm_denoise_step(model.handle, b.handle, dev_i32(tok), dev_u8(mask), W, out_i, out_c)
    torch.cuda.synchronize()
    np.testing.assert_allclose(conf, out_c.cpu().numpy(), rtol=1e-5)
    assert a.prefix_len == b.prefix_len == P0
    # block only == append
    _merged(model, a, [], [], blk, [], [])
    dl.dllm_append_prefix_kv(model.handle, b.handle, dev_i32(blk), B)
    torch.cuda.synchronize()
    assert a.prefix_len == b.prefix_len == P0 + B
    for x, y in zip(_cache(a, P0 + B), _cache(b, P0 + B)):
        np.testing.assert_allclose(x, y, atol=1e-6, rtol=1e-5)
    # refresh only == refresh
    _, _, rids, rconf = _merged(model, a, ref_pos, ref_new, [], [], [])
    r_i = torch.empty(3, dtype=torch.int32, device="cuda")
    r_c = torch.empty(3, device="cuda")
    dl.dllm_refresh_kv(model.handle, b.handle, dev_i32(ref_pos), dev_i32(ref_new), 3, r_i, r_c)
    torch.cuda.synchronize()
    np.testing.assert_allclose(rconf, r_c.cpu().numpy(), rtol=1e-5)
    np.testing.assert_array_equal(rids, r_i.cpu().numpy())
    for x, y in zip(_cache(a, P0 + B), _cache(b, P0 + B)):
        np.testing.assert_allclose(x, y, atol=1e-6, rtol=1e-5)
    a.close()
    b.close()
    model.close()


def test_merged_validation():
    sh = synth.MICRO
    model, _, _ = build_pair(sh, "f32", max_window=64, max_pos=512, oracle_too=False)
    kv = dl.KVCache(model, 100)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(np.arange(40) % 70), 40)
    blk = dev_i32(np.arange(32) % 70)
    tok = dev_i32(np.zeros(40))
    print("case: merged validation", flush=True)
    cases = [
        (dict(ref=[3, 3]), dl.DLLM_E_INVAL),                         # duplicate refresh positions
        (dict(ref=[40]), dl.DLLM_E_INVAL),                           # not in the prefix
        (dict(blk=32, W=40), dl.DLLM_E_INVAL),                       # 72 rows > max_window
        (dict(), dl.DLLM_E_INVAL),                                   # no rows
        (dict(blk=32, W=30), dl.DLLM_E_CAPACITY),                    # 40 + 32 + 30 > 100
    ]
    for c, code in cases:
        ref = c.get("ref", [])
        n_ref, n_blk, W = len(ref), c.get("blk", 0), c.get("W", 0)
        with pytest.raises(dl.DllmError) as e:
            dl.dllm_step_merged(model.handle, kv.handle, dev_i32(ref) if ref else None,
                                dev_i32(np.zeros(len(ref))) if ref else None, n_ref, blk if n_blk else None, n_blk,
                                tok if W else None, None, W)
        assert e.value.code == code, c
    assert kv.prefix_len == 40
    kv.close()
    model.close()
