"""Shared helpers of the GPU parity tests: build a library model and the oracle
from the same seeded weights, run both, compare."""
import numpy as np

import oracle
import synth

GLOBALS = ("embed", "lm_head", "final_norm")


def weight_dtype(dtype: str) -> str:
    return "f32" if dtype == "f32" else "bf16"


def build_pair(shape, dtype: str, max_window: int = 64, max_pos: int = 1024, seed: int = 0, oracle_too=True):
    """(library Model, OracleModel or None, host weights) from the same seeded draws."""
    import paper_2606_13740_amd as dl

    w = synth.all_weights(shape, weight_dtype(dtype), seed)
    model = dl.Model(shape, dtype, {k: w[k] for k in GLOBALS}, lambda l: w["layers"][l],
                     max_window=max_window, max_pos=max_pos)
    om = oracle.OracleModel(shape, w, int8=(dtype == "w8"), q4=(dtype == "q4")) if oracle_too else None
    return model, om, w


def tol(dtype: str) -> float:
    """Logit tolerance: 1e-4 for fp32 models, 5e-2 for bf16 and int8-weight models."""
    return 1e-4 if dtype == "f32" else 5e-2


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def dev_u8(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def gpu_logits(model, kv, tok, mask):
    """(logits [W, V], ids, conf) of one step through dllm_debug_logits."""
    import torch
    import paper_2606_13740_amd as dl

    W = len(tok)
    logits = torch.empty(W, model.shape.vocab, device="cuda")
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    dl.dllm_debug_logits(model.handle, kv.handle, dev_i32(tok), dev_u8(mask), W, logits, ids, conf)
    torch.cuda.synchronize()
    return logits.cpu().numpy().astype(np.float64), ids.cpu().numpy(), conf.cpu().numpy().astype(np.float64)


def gpu_step(model, kv, tok, mask):
    import torch
    import paper_2606_13740_amd as dl

    W = len(tok)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    dl.dllm_denoise_step(model.handle, kv.handle, dev_i32(tok), dev_u8(mask), W, ids, conf)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), conf.cpu().numpy().astype(np.float64)


def assert_logits_close(got, ref, atol):
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got)), "MASK column must be -inf on both sides"
    err = float(np.max(np.abs(got[fin] - ref[fin])))
    print(f"  max |dlogit| = {err:.3e} (tolerance {atol:.1e})", flush=True)
    assert err <= atol, f"max |dlogit| = {err:.3e} > {atol:.1e}"
    return err


def assert_ids_match_where_decided(got_ids, ref_logits, err_bound, ref_conf=None, got_conf=None):
    """Argmax must match wherever the oracle's top-2 logit gap exceeds 2 * err_bound
    (two logits each off by at most err_bound cannot swap), and wherever its top-2
    probability margin exceeds 1e-3.  Returns the fraction of rows decided."""
    if len(got_ids) == 0:
        return 1.0
    srt = np.sort(ref_logits, axis=-1)
    gap = srt[:, -1] - srt[:, -2]
    ref_ids = np.argmax(ref_logits, axis=-1)
    p = np.exp(ref_logits - srt[:, -1:])
    p /= p.sum(axis=-1, keepdims=True)
    ps = np.sort(p, axis=-1)
    margin = ps[:, -1] - ps[:, -2]
    decided = (gap > 2 * err_bound) | (margin > 1e-3)
    bad = np.nonzero(decided & (got_ids != ref_ids))[0]
    assert len(bad) == 0, f"argmax differs on decided rows {bad.tolist()}"
    return float(decided.mean())


def assert_commit_matches_where_decided(got_pos, ref_pos, conf_ref, mask_before, seg, k, rel_bound):
    """The committed set must match where the k-th and (k+1)-th confidences of the
    oracle differ by more than the relative bound."""
    cand = [p for p in range(seg[0], seg[0] + seg[1]) if mask_before[p]]
    c = sorted((conf_ref[p] for p in cand), reverse=True)
    if len(c) <= k or c[k - 1] - c[k] > rel_bound * c[k - 1]:
        assert set(got_pos) == set(ref_pos), (sorted(got_pos), sorted(ref_pos))
        return True
    return False
