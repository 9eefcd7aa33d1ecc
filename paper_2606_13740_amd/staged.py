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

Re-prediction of a tracked position (a reading of the Sparse Cache Refresh
passage, which recomputes confidence, identity and KV): the position is
refreshed with the MASK id, which yields the model's (id, conf) for it in the
current context; it becomes stable with that id if conf >= theta_stable, takes
that id but stays visible if conf >= theta_visible, and keeps its id otherwise;
then the chosen ids are written back with a second refresh, so the cache holds
their K/V.
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
        """Re-predict every tracked visible position of the prefix (in chunks of at most
        max_window rows, each chunk one re-prediction refresh and one write-back).
        Returns (positions that became stable, {position: id written back})."""
        became_stable, chosen = [], {}
        pos_all = sorted(self.tracked)
        for c0 in range(0, len(pos_all), self.max_rows):
            pos = np.array(pos_all[c0:c0 + self.max_rows], dtype=np.int32)
            n = len(pos)
            d_pos = torch.from_numpy(pos).to(self.dev)
            rid = torch.empty(n, dtype=torch.int32, device=self.dev)
            rconf = torch.empty(n, device=self.dev)
            masked = torch.full((n,), self.mask_id, dtype=torch.int32, device=self.dev)
            dllm_refresh_kv(self.model.handle, self.kv.handle, d_pos, masked, n, rid, rconf, self.stream)
            ids, conf = rid.cpu().numpy(), rconf.cpu().numpy()
            new = np.empty(n, dtype=np.int32)
            for j, p in enumerate(pos):
                p = int(p)
                if conf[j] >= np.float32(self.ts):
                    new[j] = ids[j]
                    became_stable.append(p)
                elif conf[j] >= np.float32(self.tv):
                    new[j] = ids[j]
                else:
                    new[j] = self.tracked[p]
            dllm_refresh_kv(self.model.handle, self.kv.handle, d_pos, torch.from_numpy(new).to(self.dev), n,
                            None, None, self.stream)
            for j, p in enumerate(pos):
                self.tracked[int(p)] = int(new[j])
                chosen[int(p)] = int(new[j])
        for p in became_stable:
            del self.tracked[p]
        return became_stable, chosen


