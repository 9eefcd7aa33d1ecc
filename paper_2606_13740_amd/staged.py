"""Block-wise generation with staged token stabilisation: the host side.

System Design, "Staged Token Stabilization" and "Sparse Cache Refresh": each
generated position is invisible (masked), visible (exposed as context, still
revisable) or stable.  Within a block, dllm_commit_staged promotes positions by
the visibility / stability thresholds (or the most confident one); a completed
block is appended to the prefix cache with its visible tokens in it, and those
stay tracked: between blocks they are re-predicted through the sparse refresh
and merged before the next step (delayed merge).  The host owns the states and
the tracked set (the Implementation section gives token-state transitions and
refresh candidates to the host runtime); every arithmetic step runs in the
library.

Re-prediction of the tracked positions (a reading of the Staged Token
Stabilization and Sparse Cache Refresh passages: confidence, identity and KV of
tracked visible tokens are recomputed sparsely until they pass the stability
threshold), block by block in block order: all tracked positions of a block are
refreshed at once with the MASK id, which yields the model's (id, conf) for each
in the current context; conf >= theta_stable -> that id and the position becomes
stable (no longer tracked), conf >= theta_visible -> that id, still visible,
otherwise it keeps its id; the chosen ids are written back with a second refresh
before the next block is re-predicted.  The decisions therefore depend only on the
tracked set and the cache, not on how many rows one call may carry.  A block's
write-back and the next block's re-prediction share one refresh call when they fit
(a row of block b attends only up to the end of block b, so it is unaffected by
the next block's rows in the same call).
"""
import numpy as np
import torch

from . import (DLLM_TOKEN_STABLE, DLLM_TOKEN_VISIBLE, dllm_append_prefix_kv, dllm_commit_staged, dllm_denoise_step,
               dllm_refresh_kv)


class StagedGenerator:
    def __init__(self, model, kv, theta_visible: float = 0.7, theta_stable: float = 0.9, stream=None,
                 device: str = "cuda"):
        self.model, self.kv = model, kv
        self.tv, self.ts = float(theta_visible), float(theta_stable)
        self.stream, self.dev = stream, device
        sh = model.shape
        self.B, self.mask_id = sh.block, sh.mask_id
        self.max_rows = model.cfg.max_window
        if self.max_rows < self.B:
            raise ValueError("staged generation needs max_window >= the block size")
        self.tracked = {}             # prefix position -> current id of a visible token
        self.steps = []               # denoising steps per block
        self.promoted = []            # positions promoted per step (host copies, for inspection)

    def _sync(self):
        (torch.cuda.current_stream() if self.stream is None else self.stream).synchronize()

    def block(self):
        """Decode one block to completion and append it; returns (ids, states) on the host."""
        B, dev = self.B, self.dev
        tok = torch.full((B,), self.mask_id, dtype=torch.int32, device=dev)
        mask = torch.ones(B, dtype=torch.uint8, device=dev)
        state = torch.zeros(B, dtype=torch.uint8, device=dev)
        ids = torch.empty(B, dtype=torch.int32, device=dev)
        conf = torch.empty(B, device=dev)
        prom = torch.empty(B, dtype=torch.int32, device=dev)
        nprom = torch.zeros(1, dtype=torch.int32, device=dev)
        h = self.model.handle
        for step in range(B):          # each step promotes at least one position
            dllm_denoise_step(h, self.kv.handle, tok, mask, B, ids, conf, self.stream)
            dllm_commit_staged(conf, ids, tok, mask, state, 0, B, self.tv, self.ts, prom, nprom, self.stream)
            self._sync()
            n = int(nprom.item())
            self.promoted.append(prom[:n].cpu().numpy())
            if not bool(mask.any()):
                break
        self.steps.append(step + 1)
        P = self.kv.prefix_len
        dllm_append_prefix_kv(h, self.kv.handle, tok, B, self.stream)
        st = state.cpu().numpy()
        t = tok.cpu().numpy()
        for i in np.flatnonzero(st == DLLM_TOKEN_VISIBLE):
            self.tracked[P + int(i)] = int(t[i])
        return t, st

    def refresh_visible(self):
        """Re-predict every tracked visible position of the prefix, block by block.
        Returns (positions that became stable, ascending; {position: id written back})."""
        P0, B, mask_id, dev = self.kv.prompt_len, self.B, self.mask_id, self.dev
        h, kvh = self.model.handle, self.kv.handle
        by_block = {}
        for p in sorted(self.tracked):
            by_block.setdefault((p - P0) // B, []).append(p)
        became_stable, chosen = [], {}
        wb_pos, wb_ids = [], []          # the previous block's write-back, not issued yet

        def refresh(pos, ids, want_out):
            n = len(pos)
            d_pos = torch.tensor(pos, dtype=torch.int32, device=dev)
            d_ids = torch.tensor(ids, dtype=torch.int32, device=dev)
            rid = torch.empty(n, dtype=torch.int32, device=dev) if want_out else None
            rconf = torch.empty(n, device=dev) if want_out else None
            dllm_refresh_kv(h, kvh, d_pos, d_ids, n, rid, rconf, self.stream)
            return rid, rconf

        for b in sorted(by_block):
            pos = by_block[b]
            if len(wb_pos) + len(pos) > self.max_rows and wb_pos:
                refresh(wb_pos, wb_ids, False)
                wb_pos, wb_ids = [], []
            rid, rconf = refresh(wb_pos + pos, wb_ids + [mask_id] * len(pos), True)
            self._sync()
            ids = rid.cpu().numpy()[len(wb_pos):]
            conf = rconf.cpu().numpy()[len(wb_pos):]
            new = []
            for j, p in enumerate(pos):
                c = np.float32(conf[j])
                if c >= np.float32(self.ts):
                    new.append(int(ids[j]))
                    became_stable.append(p)
                elif c >= np.float32(self.tv):
                    new.append(int(ids[j]))
                else:
                    new.append(self.tracked[p])
            for p, t in zip(pos, new):
                self.tracked[p] = t
                chosen[p] = t
            wb_pos, wb_ids = pos, new
        if wb_pos:
            refresh(wb_pos, wb_ids, False)
        for p in became_stable:
            del self.tracked[p]
        return sorted(became_stable), chosen
