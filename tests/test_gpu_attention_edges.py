"""Attention edge cases on the GPU against the float64 oracle.

- Cache rows past the key count T holding NaN bit patterns.  Rows at and past T are
  never written by the step that reads them (its window ends at T, and a caller-owned
  cache buffer may hold anything there), and 0 * NaN is NaN in an MFMA: the V^T values
  of keys past T must be zeroed where the block holding T is staged, and their
  scores masked.  Key counts off the 32-key block grid put T inside a block, for the
  prompt's attention, the 32-row window (one key group) and the 64-row window (two
  key groups taking alternate blocks, only one of which holds T).  The results must
  be bit-identical to those over a zero-filled cache, and match the oracle.
- Wide score ranges: W_q and W_k scaled by 2^5 each (scores ~2^10 larger, a spread
  of tens of units in the log2 domain), so that the lazily rescaled softmax maximum
  moves in the middle of a key split, not only on a row's first block.  The fp16
  cache's rounding then moves the scores by ~2^10 times more too (7e-2 off the exact
  oracle at 64 rows, the same as a softmax rescaled on every block), so these cases
  compare with the oracle storing its K/V in fp16 as well.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import GLOBALS, assert_ids_match_where_decided, assert_logits_close, dev_i32, gpu_logits, tol

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402

SH = synth.SMALL_BF16          # 2 heads of 128: the fp16 MFMA attention


def _model(w, max_pos=1024):
    return dl.Model(SH, "bf16", {k: w[k] for k in GLOBALS}, lambda l: w["layers"][l], max_window=64,
                    max_pos=max_pos)


def _scale_qk(w, log2c):
    """Multiplies W_q and W_k of every layer by 2^log2c (exact on bf16 bit patterns)."""
    for lw in w["layers"]:
        for n in ("wq", "wk"):
            f = synth.bf16_bits_to_f32(lw[n]) * np.float32(2.0 ** log2c)
            lw[n] = (f.view(np.uint32) >> 16).astype(np.uint16)
    return w


def _run(model, P, W, masked, fill):
    """Prefill P prompt ids and one step over a W-row window with the cache buffer
    first filled with `fill` (int16 bit pattern); returns the step's (logits, ids, conf)."""
    kv = dl.KVCache(model, P + W)
    kv.buf.fill_(fill)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(SH, P)), P)
    tok, mask = synth.window(SH, W, masked)
    out = gpu_logits(model, kv, tok, mask)
    kv.close()
    return out


def _oracle(w, P, W, masked, fp16=False):
    om = oracle.OracleModel(SH, w)
    okv = oracle.OracleKV(SH, P + W, fp16=fp16)
    oracle.prefill(om, okv, synth.prompt_ids(SH, P))
    tok, mask = synth.window(SH, W, masked)
    return oracle.denoise_step(om, okv, tok, mask)


@pytest.mark.parametrize("P,W", [(69, 32), (69, 64), (100, 27)])
def test_nan_past_key_count_never_reaches_the_output(P, W):
    print(f"case: NaN-filled cache, prefix {P}, window {W} (T = {P + W})", flush=True)
    assert (P + W) % 32 != 0 and P % 32 != 0
    w = synth.all_weights(SH, "bf16")
    model = _model(w)
    masked = list(range(W // 4, W))
    lz, iz, cz = _run(model, P, W, masked, 0)
    ln, i_n, cn = _run(model, P, W, masked, -1)        # 0xFFFF: an fp16 NaN in every cache slot
    assert np.all(np.isfinite(ln[:, :SH.mask_id]))
    np.testing.assert_array_equal(ln, lz)
    np.testing.assert_array_equal(i_n, iz)
    np.testing.assert_array_equal(cn, cz)
    ref = _oracle(w, P, W, masked)
    err = assert_logits_close(ln, ref.logits, tol("bf16"))
    assert_ids_match_where_decided(i_n, ref.logits, err)
    model.close()


@pytest.mark.parametrize("P,W", [(300, 32), (200, 64), (69, 64)])
def test_wide_score_range_matches_oracle(P, W):
    """Scores spread over tens of log2 units: the lazily rescaled maximum moves within
    splits (and within the prompt's unsplit key loops), and every probability stays
    within the rescale slack."""
    print(f"case: W_q, W_k x 2^5, prefix {P}, window {W}", flush=True)
    w = _scale_qk(synth.all_weights(SH, "bf16"), 5)
    model = _model(w)
    masked = list(range(W // 4, W))
    logits, ids, conf = _run(model, P, W, masked, 0)
    ref = _oracle(w, P, W, masked, fp16=True)
    err = assert_logits_close(logits, ref.logits, tol("bf16"))
    frac = assert_ids_match_where_decided(ids, ref.logits, err)
    print(f"  argmax decided on {frac:.0%} of rows", flush=True)
    np.testing.assert_allclose(conf, ref.conf, rtol=0.2)
    model.close()
