"""Multi-block speculative decoding: the window policy (oracle side).

TEST INFRASTRUCTURE, like the rest of this package: only the tests, the smoke
check and the benchmark's CPU-baseline leg may use it.

System Design, "Multi-Block Speculative Decoding".  The decoding window, not the
block, is the unit one forward runs over; the block stays the unit of left-to-right
commitment.  Window rows past the current block are drafts: their predictions are
recorded, they are never committed while their block is not current, and they
never become prefix.  Two strategies move the window:
  * continuous sliding: the window keeps its size and moves right as committed
    positions at its left edge are done with;
  * adaptive lookahead: once few masked positions remain in the current block, the
    window grows by as many extra rows as a profiled latency table allows within an
    allowance.
When a block becomes current, its drafts are re-evaluated and accepted only if they
meet the acceptance criterion.

Readings taken where the paper is silent (the GPU driver takes the same ones):
  * the window's left edge moves past a committed position only after a step that
    ran with that position's committed id (a position committed at step t is passed
    at the end of step t + 1 at the earliest); the K/V that step wrote are kept, and
    when the edge passes the end of the current block the block becomes prefix
    without a recompute pass;
  * commitment in the current block: the k most confident masked positions per step
    (ties -> lower position), as the top-k commit;
  * a draft is accepted, in the first step its block is current, if that step
    predicts the same id as the draft recorded and its confidence reaches
    theta_accept (fp32 comparison); accepted positions are committed then;
  * a draft record is the id the latest step predicted for a masked position past
    the current block; committed positions hold no record (-1);
  * lookahead: with r masked positions left in the current block and r <= tau, the
    window takes the largest row count R in the latency table with
    latency(R) <= (1 + allowance) * latency(Wn); the window never runs past the
    last generated position.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from .model import OracleKV, OracleModel, commit, denoise_window


def accept_drafts(conf: np.ndarray, pred: np.ndarray, draft_id: np.ndarray, tok: np.ndarray, mask: np.ndarray,
                  theta: float) -> np.ndarray:
    """Accept the drafts of a block that has become current: every masked position
    whose draft record equals this step's prediction with conf >= theta (fp32) is
    committed.  Arrays are position-aligned; tok / mask are updated in place.
    Returns the accepted positions, ascending."""
    c, th = np.asarray(conf, dtype=np.float32), np.float32(theta)
    acc = [i for i in range(len(c)) if mask[i] == 1 and draft_id[i] >= 0 and pred[i] == draft_id[i] and c[i] >= th]
    for i in acc:
        tok[i] = pred[i]
        mask[i] = 0
    return np.array(acc, dtype=np.int32)


def record_drafts(pred: np.ndarray, mask: np.ndarray, draft_id: np.ndarray) -> None:
    """Record this step's predictions of the masked draft positions (-1 elsewhere)."""
    for i in range(len(pred)):
        draft_id[i] = pred[i] if mask[i] == 1 else -1


def lookahead_rows(Wn: int, remaining: int, tau: int, table: Sequence[Tuple[int, float]], allowance: float) -> int:
    """Window rows for the next step: Wn, or the largest profiled row count whose
    latency stays within (1 + allowance) of Wn's once <= tau masked positions remain."""
    if remaining > tau:
        return Wn
    lat = dict(table)
    base = lat[Wn]
    best = Wn
    for r, t in table:
        if r > best and t <= (1.0 + allowance) * base:
            best = r
    return best


def generate(model: OracleModel, kv: OracleKV, n_gen: int, Wn: int, k: int, tau: int,
             table: Sequence[Tuple[int, float]], allowance: float, theta_accept: float,
             max_steps: int = 100000) -> Dict:
    """Decode n_gen positions after the prefix (a multiple of the block size) with
    the window policy.  Returns the final ids and a per-step trace."""
    sh = model.shape
    B, MASK = sh.block, sh.mask_id
    start = kv.prefix_len
    end = start + n_gen
    assert n_gen % B == 0 and end <= kv.capacity
    tok = np.full(n_gen, MASK, dtype=np.int64)
    mask = np.ones(n_gen, dtype=np.uint8)
    commit_step = np.full(n_gen, -1)
    draft_id = np.full(n_gen, -1, dtype=np.int64)
    P, w0, fresh = start, start, False
    trace: List[Dict] = []
    for t in range(max_steps):
        cur = slice(P - start, P - start + B)
        remaining = int(mask[cur].sum())
        R = lookahead_rows(Wn, remaining, tau, table, allowance)
        W = min(R, end - w0)
        a, b = w0 - start, w0 - start + W
        so = denoise_window(model, kv, w0, tok[a:b], mask[a:b])
        cur_end = min(P + B, w0 + W) - w0                      # window rows of the current block
        accepted = np.zeros(0, dtype=np.int32)
        if fresh:
            accepted = accept_drafts(so.conf[:cur_end], so.ids[:cur_end], draft_id[a:a + cur_end],
                                     tok[a:a + cur_end], mask[a:a + cur_end], theta_accept)
            fresh = False
        seg_tok, seg_mask = tok[a:a + cur_end], mask[a:a + cur_end]
        committed = commit(so.conf[:cur_end], so.ids[:cur_end], seg_tok, seg_mask, 0, cur_end, k)
        for i in list(accepted) + list(committed):
            commit_step[a + i] = t
        if W > cur_end:                                        # drafts past the current block
            record_drafts(so.ids[cur_end:], mask[a + cur_end:b], draft_id[a + cur_end:b])
        draft_id[a:a + cur_end][mask[a:a + cur_end] == 0] = -1
        while w0 < P + B and mask[w0 - start] == 0 and commit_step[w0 - start] < t:
            w0 += 1
        settled = False
        if w0 == P + B:
            P += B
            kv.prefix_len = P
            fresh, settled = True, True
        trace.append(dict(step=t, w0=a + start, W=W, R=R, remaining=remaining,
                          committed=[a + int(i) + start for i in committed],
                          accepted=[a + int(i) + start for i in accepted], settled=settled, prefix=P))
        if P == end:
            break
    return dict(tok=tok, trace=trace)
