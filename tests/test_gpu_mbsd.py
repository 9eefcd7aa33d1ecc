"""Multi-block speculative decoding on the GPU against the oracle.

The slid-window step is compared with the oracle's (and with the fixed point it
must reproduce when nothing changed); draft acceptance and recording bit-exactly;
the GPU driver's whole run is replayed in the oracle step by step: the same
inputs give the same confidences within tolerance, the GPU's confidences give
the same decisions under the oracle's policy functions, the trace keeps the
policy's invariants, and the final cache matches.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_ids_match_where_decided, build_pair, dev_i32, dev_u8
from oracle import mbsd as ombsd

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402


def _win(model, kv, w0, tok, mask):
    W = len(tok)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    dl.dllm_denoise_window(model.handle, kv.handle, w0, dev_i32(tok), dev_u8(mask), W, ids, conf)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), conf.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_slid_window_matches_oracle(dtype):
    sh = synth.TINY if dtype == "f32" else synth.SMALL_BF16
    atol, rtol = (1e-4, 1e-3) if dtype == "f32" else (5e-2, 0.1)
    model, om, _ = build_pair(sh, dtype, max_pos=512)
    P0, W, s = 64, 24, 9
    kv = dl.KVCache(model, P0 + 40)
    okv = oracle.OracleKV(sh, P0 + 40)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    oracle.prefill(om, okv, prompt)
    ids = synth.uniform_ids(7, 1, W, sh.mask_id)
    mask = np.zeros(W, np.uint8)
    mask[15:] = 1
    print(f"case: slid window {dtype}", flush=True)
    i1, c1 = _win(model, kv, P0, ids, mask)
    i2, c2 = _win(model, kv, P0 + s, ids[s:], mask[s:])
    oracle.denoise_window(om, okv, P0, ids, mask)
    so = oracle.denoise_window(om, okv, P0 + s, ids[s:], mask[s:])
    np.testing.assert_allclose(c2, so.conf, rtol=rtol)
    assert_ids_match_where_decided(i2, so.logits, atol)
    np.testing.assert_allclose(c2, c1[s:], rtol=1e-5 if dtype == "f32" else 1e-2)   # nothing changed: fixed point
    assert kv.prefix_len == P0
    with pytest.raises(dl.DllmError) as e:
        _win(model, kv, P0 - 1, ids, mask)
    assert e.value.code == dl.DLLM_E_INVAL
    kv.close()
    model.close()


@pytest.mark.parametrize("n", [1, 33, 1024])
def test_accept_and_record_drafts_bit_exact(n):
    rng = np.random.default_rng(n)
    for case in range(20):
        conf = rng.random(n).astype(np.float32)
        if case % 3 == 0:
            conf = (np.round(conf * 4) / 4).astype(np.float32)
        pred = rng.integers(0, 5, n).astype(np.int32)
        draft = np.where(rng.random(n) < 0.7, rng.integers(0, 5, n), -1).astype(np.int32)
        mask = (rng.random(n) < 0.6).astype(np.uint8)
        tok = np.where(mask == 1, 999, rng.integers(0, 5, n)).astype(np.int32)
        theta = float(rng.choice([0.0, 0.5, 1.5]))
        d_tok, d_mask = dev_i32(tok), dev_u8(mask)
        apos = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        nacc = torch.zeros(1, dtype=torch.int32, device="cuda")
        dl.dllm_accept_drafts(torch.from_numpy(conf).cuda(), dev_i32(pred), dev_i32(draft), d_tok, d_mask, n, theta,
                              apos, nacc)
        rec = torch.full((n,), 5, dtype=torch.int32, device="cuda")
        dl.dllm_record_drafts(dev_i32(pred), d_mask, rec, n)
        torch.cuda.synchronize()
        t2, m2 = tok.copy(), mask.copy()
        want = ombsd.accept_drafts(conf, pred, draft, t2, m2, theta)
        r2 = np.full(n, 5)
        ombsd.record_drafts(pred, m2, r2)
        np.testing.assert_array_equal(d_tok.cpu().numpy(), t2)
        np.testing.assert_array_equal(d_mask.cpu().numpy(), m2)
        np.testing.assert_array_equal(apos.cpu().numpy()[:int(nacc.item())], want)
        np.testing.assert_array_equal(rec.cpu().numpy(), r2)


@pytest.mark.parametrize("sls", [False, True])
def test_driver_run_replays_in_the_oracle(sls):
    from paper_2606_13740_amd.mbsd import MBSDGenerator

    sh = synth.TINY
    model, om, _ = build_pair(sh, "f32", max_pos=512)
    B, P0, n_gen, k, tau = sh.block, 64, 2 * sh.block, 2, 4
    table = [(32, 1.0), (40, 1.03), (48, 1.06), (64, 1.3)]
    kv = dl.KVCache(model, P0 + n_gen)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    print(f"case: MBSD driver, tiny fp32, 2 blocks, sls {sls}", flush=True)
    gen = MBSDGenerator(model, kv, n_gen, window=32, k=k, tau=tau, latency_table=table, allowance=0.1,
                        theta_accept=0.0, record=True, sls=sls)
    final = gen.run()
    tr = gen.trace
    assert np.all(final != sh.mask_id) and kv.prefix_len == P0 + n_gen
    assert any(e["R"] > 32 for e in tr), "lookahead never triggered"
    okv = oracle.OracleKV(sh, P0 + n_gen)
    oracle.prefill(om, okv, prompt)
    draft = np.full(n_gen, -1)
    P, fresh, done = P0, False, set()
    for e in tr:
        w0, W = e["w0"], e["W"]
        a = w0 - P0
        assert w0 >= P and e["W"] == min(e["R"], P0 + n_gen - w0)
        so = oracle.denoise_window(om, okv, w0, e["tok"], e["mask"])
        rows = np.flatnonzero(e["mask"]) if sls else np.arange(W)      # rows with an output
        np.testing.assert_allclose(e["conf"][rows], so.conf[rows], rtol=1e-3)
        assert_ids_match_where_decided(e["ids"][rows], so.logits[rows], 1e-4)
        if sls:
            off = np.flatnonzero(e["mask"] == 0)
            assert np.all(e["ids"][off] == -1) and np.all(e["conf"][off] == 0.0)
        # the GPU's confidences under the oracle's policy functions give the same decisions
        cur = min(P + B, w0 + W) - w0
        tok, mask = e["tok"].astype(np.int64).copy(), e["mask"].copy()
        acc = np.zeros(0, np.int32)
        if fresh:
            acc = ombsd.accept_drafts(e["conf"][:cur], e["ids"][:cur], draft[a:a + cur], tok[:cur], mask[:cur], 0.0)
        com = oracle.commit(e["conf"][:cur].astype(np.float64), e["ids"][:cur], tok, mask, 0, cur, k)
        assert (w0 + acc).tolist() == e["accepted"] and (w0 + com).tolist() == e["committed"]
        if W > cur:
            ombsd.record_drafts(e["ids"][cur:], mask[cur:], draft[a + cur:a + W])
        for p in e["accepted"] + e["committed"]:
            assert P <= p < P + B and p not in done
            done.add(p)
        fresh = False
        if e["settled"]:
            P, fresh = P + B, True
            okv.prefix_len = P
        assert e["prefix"] == P
    assert done == set(range(P0, P0 + n_gen))
    K, Vt = kv.views()
    n = P0 + n_gen
    np.testing.assert_allclose(K[:, :, :n].cpu().numpy(), np.transpose(okv.K[:, :n], (0, 2, 1, 3)), atol=2e-4, rtol=0)
    np.testing.assert_allclose(np.swapaxes(Vt[:, :, :, :n].cpu().numpy(), 2, 3),
                               np.transpose(okv.V[:, :n], (0, 2, 1, 3)), atol=2e-4, rtol=0)
    kv.close()
    model.close()
