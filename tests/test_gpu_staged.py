"""Staged token stabilisation on the GPU (dllm_commit_staged) against the oracle.

Both sides compare the same float32 confidences with the same float32 thresholds, so
every decision, the promoted positions, the new ids, masks and states must match
bit-exactly.  The loop test runs the kernel on the confidences the GPU step itself
produced, over whole blocks, with thresholds drawn from that step's confidence
quantiles so that threshold promotions, fallback promotions and stable transitions
all occur.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import build_pair, dev_i32, dev_u8, gpu_step

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402


def _dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _run_gpu(conf, pred, tok, mask, state, b, ln, tv, ts):
    d_tok, d_mask, d_state = dev_i32(tok), dev_u8(mask), dev_u8(state)
    prom = torch.full((max(ln, 1),), -1, dtype=torch.int32, device="cuda")
    nprom = torch.zeros(1, dtype=torch.int32, device="cuda")
    dl.dllm_commit_staged(_dev_f32(conf), dev_i32(pred), d_tok, d_mask, d_state, b, ln, tv, ts, prom, nprom)
    torch.cuda.synchronize()
    n = int(nprom.item())
    return (d_tok.cpu().numpy(), d_mask.cpu().numpy(), d_state.cpu().numpy(), prom.cpu().numpy()[:n])


@pytest.mark.parametrize("n", [1, 7, 64, 100, 1024])
def test_staged_commit_matches_oracle(n):
    rng = np.random.default_rng(n)
    for case in range(30):
        print(f"case: n {n} #{case}", flush=True)
        conf = rng.random(n).astype(np.float32)
        if case % 3 == 0:
            conf = (np.round(conf * 8) / 8).astype(np.float32)          # ties
        if case % 5 == 0:
            conf[:] = 0.0                                                 # all zero: fallback to the lowest position
        state = rng.integers(0, 3, n).astype(np.uint8)
        if case % 4 == 0:
            state[:] = oracle.IV
        mask = (state == oracle.IV).astype(np.uint8)
        pred = rng.integers(0, 126000, n).astype(np.int32)
        tok = np.where(mask == 1, 126463, rng.integers(0, 126000, n)).astype(np.int32)
        same = (mask == 0) & (rng.random(n) < 0.5)          # visible rows predicting their held id
        tok[same] = pred[same]
        b = int(rng.integers(0, n))
        ln = int(rng.integers(1, n - b + 1))
        tv = float(rng.choice([0.0, 0.25, 0.7, 1.5]))
        ts = float(rng.choice([0.3, 0.9, 2.0]))
        got = _run_gpu(conf, pred, tok, mask, state, b, ln, tv, ts)
        t2, m2, s2 = tok.copy(), mask.copy(), state.copy()
        want = oracle.commit_staged(conf, pred, t2, m2, s2, b, ln, tv, ts)
        np.testing.assert_array_equal(got[0], t2)
        np.testing.assert_array_equal(got[1], m2)
        np.testing.assert_array_equal(got[2], s2)
        np.testing.assert_array_equal(got[3], want)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_staged_generation_loop(dtype):
    """Whole blocks decoded with staged commits on the GPU's own confidences; the
    kernel's decisions equal the oracle's on those confidences at every step, every
    step promotes at least one position while any is invisible, and states only move
    forward."""
    sh = synth.TINY if dtype == "f32" else synth.SMALL_BF16
    model, _, _ = build_pair(sh, dtype, max_pos=512, oracle_too=False)
    P0, B = 64, sh.block
    kv = dl.KVCache(model, P0 + 2 * B)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(sh, P0)), P0)
    for blk in range(2):
        tok, mask = synth.window(sh, B, range(B))
        state = np.zeros(B, np.uint8)
        for step in range(B):
            print(f"case: {dtype} block {blk} step {step}", flush=True)
            ids, conf = gpu_step(model, kv, tok, mask)
            tv, ts = (float(np.quantile(conf, 0.8)), float(np.quantile(conf, 0.95))) if step % 2 == 0 else (2.0, 3.0)
            got = _run_gpu(conf, ids, tok, mask, state, 0, B, tv, ts)
            t2, m2, s2 = tok.copy(), mask.copy(), state.copy()
            want = oracle.commit_staged(conf, ids, t2, m2, s2, 0, B, tv, ts)
            np.testing.assert_array_equal(got[0], t2)
            np.testing.assert_array_equal(got[1], m2)
            np.testing.assert_array_equal(got[2], s2)
            np.testing.assert_array_equal(got[3], want)
            assert len(want) >= 1 and np.all(s2 >= state)
            tok, mask, state = t2, m2, s2
            if not mask.any():
                break
        assert not mask.any()
        dl.dllm_append_prefix_kv(model.handle, kv.handle, dev_i32(tok), B)


@pytest.mark.parametrize("max_window", [64, 32])
def test_staged_generator_matches_oracle_repredict(max_window):
    """The host driver (paper_2606_13740_amd.staged): blocks decoded with staged
    commits and appended with their visible tokens, then the re-prediction of every
    tracked position.  The oracle replays the same appends and runs its own
    re-prediction rule (oracle.repredict_tracked) from the same tracked set: the
    positions that became stable, the ids written back and the whole cache must match.
    With max_window 64 the driver shares one refresh between a block's write-back and
    the next block's re-prediction; with 32 it cannot, and the result is the same."""
    from paper_2606_13740_amd.staged import StagedGenerator

    sh = synth.TINY
    model, om, _ = build_pair(sh, "f32", max_window=max_window, max_pos=512)
    P0, B, nb = 64, sh.block, 3
    kv = dl.KVCache(model, P0 + nb * B)
    prompt = synth.prompt_ids(sh, P0)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(prompt), P0)
    okv = oracle.OracleKV(sh, P0 + nb * B)
    oracle.prefill(om, okv, prompt)
    tok0, mask0 = synth.window(sh, B, range(B))
    _, conf0 = gpu_step(model, kv, tok0, mask0)
    gen = StagedGenerator(model, kv, theta_visible=float(np.quantile(conf0, 0.6)),
                          theta_stable=float(np.quantile(conf0, 0.9)))
    ts_blocks = [2.0, gen.ts, gen.ts]        # block 0 keeps every promoted token visible
    n_prom = 0
    for b in range(nb):
        print(f"case: staged generator block {b}, max_window {max_window}", flush=True)
        gen.ts = ts_blocks[b]
        t, st = gen.block()
        assert np.all(st != oracle.IV) and gen.steps[-1] <= B
        block_prom = gen.promoted[n_prom:]
        n_prom = len(gen.promoted)
        assert all(len(p) >= 1 for p in block_prom)
        assert sorted(np.concatenate(block_prom).tolist()) == list(range(B))     # each position once
        oracle.append_block(om, okv, t)
    assert len(gen.tracked) >= B, "block 0's tokens all stay visible"
    # re-prediction thresholds between observed confidences of the first tracked block
    first = [p for p in sorted(gen.tracked) if (p - P0) // B == (min(gen.tracked) - P0) // B]
    _, c_probe, _ = oracle.refresh(om, okv.copy(), first, [sh.mask_id] * len(first))
    c = np.sort(c_probe.astype(np.float32))
    i1, i2 = len(c) // 3, 2 * len(c) // 3
    gen.tv, gen.ts = float((c[i1 - 1] + c[i1]) / 2), float((c[i2 - 1] + c[i2]) / 2)
    tracked_before = dict(gen.tracked)
    stable, chosen = gen.refresh_visible()
    o_tracked = dict(tracked_before)
    o_stable, o_chosen = oracle.repredict_tracked(om, okv, o_tracked, gen.tv, gen.ts)
    print(f"  tracked {len(tracked_before)}, stable {len(stable)}, "
          f"changed ids {sum(chosen[p] != tracked_before[p] for p in chosen)}", flush=True)
    assert stable == o_stable
    assert chosen == o_chosen
    assert gen.tracked == o_tracked
    assert 0 < len(stable) < len(tracked_before)
    K, Vt = kv.views()
    n = okv.prefix_len
    Kg = K.cpu().numpy()[:, :, :n, :]
    Vg = np.swapaxes(Vt.cpu().numpy()[:, :, :, :n], 2, 3)
    np.testing.assert_allclose(Kg, np.transpose(okv.K[:, :n], (0, 2, 1, 3)), atol=2e-4, rtol=0)
    np.testing.assert_allclose(Vg, np.transpose(okv.V[:, :n], (0, 2, 1, 3)), atol=2e-4, rtol=0)


def test_staged_commit_keeps_a_visible_token_whose_prediction_moved():
    """The GPU kernel's stability rule is the held token's: a visible position whose
    step predicts another id stays visible at any confidence."""
    conf = np.array([0.95, 0.95, 0.95, 0.10], np.float32)
    pred = np.array([5, 6, 7, 8], np.int32)
    tok = np.array([4, 6, 99, 99], np.int32)
    mask = np.array([0, 0, 1, 1], np.uint8)
    state = np.array([oracle.V, oracle.V, oracle.IV, oracle.IV], np.uint8)
    got = _run_gpu(conf, pred, tok, mask, state, 0, 4, 0.7, 0.9)
    assert got[2].tolist() == [oracle.V, oracle.S, oracle.S, oracle.IV]
    assert got[0].tolist() == [4, 6, 7, 99] and got[1].tolist() == [0, 0, 0, 1] and got[3].tolist() == [2]
