"""Pins for the oracle's multi-block speculative decoding (window policy).

The slid window is checked against an independent full forward (PyTorch SDPA and
complex-number RoPE, from test_oracle) in the case where the slid-past rows'
cached K/V are exactly the full-sequence values; draft acceptance by its
set-algebra postconditions; the policy by invariants stated in the paper (the
window keeps its size unless lookahead is triggered, drafts are never committed
before their block is current, completed blocks become prefix, everything ends
committed).
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import mbsd
from test_oracle import micro_model, torch_forward

MICRO = synth.MICRO


def _prefilled(model, P0, cap, seed=3):
    kv = oracle.OracleKV(model.shape, cap)
    prompt = synth.uniform_ids(seed, 1, P0, model.shape.mask_id)
    oracle.prefill(model, kv, prompt)
    return kv, prompt


def test_window_at_the_prefix_is_the_step():
    model, _ = micro_model()
    kv, _ = _prefilled(model, 16, 64)
    tok, mask = synth.window(MICRO, 20, range(3, 17))
    a = oracle.denoise_step(model, kv.copy(), tok, mask)
    b = oracle.denoise_window(model, kv.copy(), 16, tok, mask)
    np.testing.assert_array_equal(a.logits, b.logits)


def test_slid_window_equals_full_forward_when_nothing_changed():
    """A first window over [P, P + W) with final ids writes the full-forward K/V of
    those rows; sliding by s and running the rest again must reproduce the full
    forward's logits for rows [P + s, P + W), and leave rows [0, P + s) alone."""
    model, w = micro_model()
    P0, W, s = 16, 24, 9
    kv, prompt = _prefilled(model, P0, 64)
    ids = synth.uniform_ids(7, 1, W, MICRO.mask_id)
    zero = np.zeros(W, np.uint8)
    oracle.denoise_window(model, kv, P0, ids, zero)
    K0, V0 = kv.K[:, :P0 + s].copy(), kv.V[:, :P0 + s].copy()
    out = oracle.denoise_window(model, kv, P0 + s, ids[s:], zero[s:])
    np.testing.assert_array_equal(kv.K[:, :P0 + s], K0)
    np.testing.assert_array_equal(kv.V[:, :P0 + s], V0)
    allowed = oracle.block_causal_allowed(P0 + W, P0, MICRO.block, window_from=P0)
    ref = torch_forward(MICRO, w, np.concatenate([prompt, ids]), allowed)
    np.testing.assert_allclose(out.logits, ref[P0 + s:], atol=1e-9, rtol=0)


@pytest.mark.parametrize("seed", range(30))
def test_accept_drafts_postconditions(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    conf = rng.random(n).astype(np.float32)
    if seed % 3 == 0:
        conf = (np.round(conf * 4) / 4).astype(np.float32)
    pred = rng.integers(0, 6, n)
    draft = np.where(rng.random(n) < 0.7, rng.integers(0, 6, n), -1)
    mask = (rng.random(n) < 0.6).astype(np.uint8)
    tok = np.where(mask == 1, 99, rng.integers(0, 6, n))
    theta = float(rng.choice([0.0, 0.3, 0.75, 1.5]))
    t2, m2 = tok.copy(), mask.copy()
    acc = mbsd.accept_drafts(conf, pred, draft, t2, m2, theta)
    want = {i for i in range(n) if mask[i] and draft[i] >= 0 and draft[i] == pred[i] and conf[i] >= np.float32(theta)}
    assert set(acc.tolist()) == want and list(acc) == sorted(acc)
    for i in range(n):
        if i in want:
            assert t2[i] == pred[i] and m2[i] == 0
        else:
            assert t2[i] == tok[i] and m2[i] == mask[i]
    if theta > 1:
        assert len(acc) == 0


def test_record_drafts_keeps_masked_predictions_only():
    pred = np.array([4, 5, 6, 7])
    mask = np.array([1, 0, 1, 0], np.uint8)
    d = np.full(4, -7)
    mbsd.record_drafts(pred, mask, d)
    assert d.tolist() == [4, -1, 6, -1]


def test_lookahead_rows():
    table = [(32, 1.0), (40, 1.04), (48, 1.09), (64, 1.3), (128, 2.5)]
    assert mbsd.lookahead_rows(32, 10, 4, table, 0.1) == 32      # not triggered
    assert mbsd.lookahead_rows(32, 4, 4, table, 0.1) == 48       # largest within 10 %
    assert mbsd.lookahead_rows(32, 0, 4, table, 0.3) == 64
    assert mbsd.lookahead_rows(32, 1, 4, table, 0.0) == 32


@pytest.mark.parametrize("k,theta", [(2, 0.0), (3, 2.0)])
def test_generate_invariants(k, theta):
    model, _ = micro_model()
    B = MICRO.block
    P0, n_gen, Wn, tau = 16, 2 * B, B, 4
    table = [(32, 1.0), (40, 1.03), (48, 1.06), (64, 1.3)]
    kv, _ = _prefilled(model, P0, P0 + n_gen)
    out = mbsd.generate(model, kv, n_gen, Wn, k, tau, table, 0.1, theta)
    tr = out["trace"]
    assert np.all(out["tok"] != MICRO.mask_id)
    assert kv.prefix_len == P0 + n_gen and tr[-1]["prefix"] == P0 + n_gen
    commit_step = {}
    P, w0, fresh = P0, P0, False
    for e in tr:
        assert e["w0"] >= w0 and e["w0"] >= P                      # the window only moves right
        w0 = e["w0"]
        assert e["R"] in (Wn, 40, 48, 64) and (e["R"] == Wn or e["remaining"] <= tau)
        assert e["W"] == min(e["R"], P0 + n_gen - w0)
        for p in e["committed"] + e["accepted"]:
            assert P <= p < P + B                                   # only the current block commits
            assert p not in commit_step
            commit_step[p] = e["step"]
        assert len(e["committed"]) <= k
        if e["accepted"]:
            assert fresh                                            # acceptance only when a block turns current
        fresh = False
        if e["settled"]:
            assert e["prefix"] == P + B
            assert all(commit_step[p] < e["step"] for p in range(P, P + B))   # ran once with its id
            P, fresh = P + B, True
        else:
            assert e["prefix"] == P
    assert sorted(commit_step) == list(range(P0, P0 + n_gen))
    if theta > 1:
        assert not any(e["accepted"] for e in tr)
