"""Multi-block speculative decoding: the host driver of the decoding window.

System Design, "Multi-Block Speculative Decoding".  A forward runs over a decoding
window rather than a block; the block stays the unit of left-to-right commitment.
This driver owns the window's placement (the Implementation section leaves
lookahead positions and denoising control to the host runtime); every arithmetic
step runs in the library: dllm_denoise_window (the forward), dllm_accept_drafts,
dllm_commit and dllm_record_drafts.

Policy (the readings of the passage this module takes):
  * the window has `window` rows and starts at the first position of the current
    block that is not yet done with; a committed position is done with after one
    step has run with its committed id, so the window's left edge passes a position
    committed at step t at the end of step t + 1 at the earliest.  The K/V that
    step wrote stay in the cache; once the edge passes the end of the current block
    that block becomes prefix (prefix_len += block) with no recompute pass;
  * rows past the current block are drafts: their predictions are recorded, never
    committed, and never become prefix while their block is not current;
  * in the first step a block is current, its drafts whose recorded id this step
    predicts again with conf >= theta_accept are committed (draft acceptance);
  * every step commits the k most confident masked positions of the current block
    that the window holds;
  * adaptive lookahead: once at most `tau` masked positions remain in the current
    block, the window takes the largest row count of the latency table whose
    latency stays within (1 + allowance) of the base window's;
  * with `sls` (selective logits skipping), only the window's masked rows get an
    LM-head output: a committed row's prediction is never used again (commits,
    acceptance and draft records read masked rows only).
"""
import numpy as np
import torch

from . import (dllm_accept_drafts, dllm_commit, dllm_denoise_window, dllm_denoise_window_sls, dllm_kv_set_prefix_len,
               dllm_record_drafts)


class MBSDGenerator:
    def __init__(self, model, kv, n_gen: int, window: int = 32, k: int = 1, tau: int = 4, latency_table=None,
                 allowance: float = 0.1, theta_accept: float = 0.9, stream=None, device: str = "cuda",
                 record: bool = False, sls: bool = True):
        sh = model.shape
        self.model, self.kv = model, kv
        self.B, self.mask_id = sh.block, sh.mask_id
        if n_gen % self.B:
            raise ValueError("n_gen must be a multiple of the block size")
        if window > model.cfg.max_window:
            raise ValueError("window larger than the model's max_window")
        self.start = kv.prefix_len
        self.end = self.start + n_gen
        self.Wn, self.k, self.tau = window, k, tau
        self.table = sorted(latency_table) if latency_table else [(window, 1.0)]
        self.allowance, self.theta = allowance, float(theta_accept)
        self.stream, self.dev, self.record, self.sls = stream, device, record, sls
        self.tok = torch.full((n_gen,), self.mask_id, dtype=torch.int32, device=device)
        self.mask = torch.ones(n_gen, dtype=torch.uint8, device=device)
        self.draft = torch.full((n_gen,), -1, dtype=torch.int32, device=device)
        self.trace = []

    def rows(self, remaining: int) -> int:
        if remaining > self.tau:
            return self.Wn
        base = dict(self.table)[self.Wn]
        cands = [r for r, t in self.table if r >= self.Wn and t <= (1.0 + self.allowance) * base]
        return max(cands + [self.Wn])

    def _sync(self):
        (torch.cuda.current_stream() if self.stream is None else self.stream).synchronize()

    def run(self):
        """Decode all n_gen positions; returns the final ids (host)."""
        B, dev = self.B, self.dev
        wmax = max(r for r, _ in self.table)
        ids = torch.empty(max(wmax, self.Wn), dtype=torch.int32, device=dev)
        conf = torch.empty(max(wmax, self.Wn), device=dev)
        cpos = torch.empty(B, dtype=torch.int32, device=dev)
        ncom = torch.zeros(1, dtype=torch.int32, device=dev)
        apos = torch.empty(B, dtype=torch.int32, device=dev)
        nacc = torch.zeros(1, dtype=torch.int32, device=dev)
        h, kvh = self.model.handle, self.kv.handle
        masked = np.ones(self.end - self.start, dtype=bool)       # host mirror of the mask
        cstep = np.full(self.end - self.start, -1)
        P, w0, fresh, t = self.start, self.start, False, 0
        while True:
            remaining = int(masked[P - self.start:P - self.start + B].sum())
            R = self.rows(remaining)
            W = min(R, self.end - w0)
            a = w0 - self.start
            if self.record:
                rec = dict(step=t, w0=w0, W=W, R=R, remaining=remaining, tok=self.tok[a:a + W].cpu().numpy(),
                           mask=self.mask[a:a + W].cpu().numpy())
            if self.sls:
                n_need = int(masked[a:a + W].sum())
                dllm_denoise_window_sls(h, kvh, w0, self.tok[a:], self.mask[a:], self.mask[a:], n_need, W, ids, conf,
                                        self.stream)
            else:
                dllm_denoise_window(h, kvh, w0, self.tok[a:], self.mask[a:], W, ids, conf, self.stream)
            cur = min(P + B, w0 + W) - w0
            acc = np.zeros(0, dtype=np.int64)
            if fresh:
                dllm_accept_drafts(conf, ids, self.draft[a:], self.tok[a:], self.mask[a:], cur, self.theta, apos,
                                   nacc, self.stream)
            dllm_commit(conf, ids, self.tok[a:], self.mask[a:], 0, cur, self.k, cpos, ncom, self.stream)
            if W > cur:
                dllm_record_drafts(ids[cur:], self.mask[a + cur:], self.draft[a + cur:], W - cur, self.stream)
            self._sync()
            if fresh:
                acc = apos[:int(nacc.item())].cpu().numpy().astype(np.int64)
                fresh = False
            com = cpos[:int(ncom.item())].cpu().numpy().astype(np.int64)
            for i in np.concatenate([acc, com]):
                masked[a + i] = False
                cstep[a + i] = t
            while w0 < P + B and not masked[w0 - self.start] and cstep[w0 - self.start] < t:
                w0 += 1
            settled = w0 == P + B
            if settled:
                P += B
                dllm_kv_set_prefix_len(kvh, P)
                fresh = True
            base = a + self.start            # absolute position of window row 0
            e = dict(step=t, w0=base, W=W, R=R, remaining=remaining, committed=(base + com).tolist(),
                     accepted=(base + acc).tolist(), settled=settled, prefix=P)
            if self.record:
                rec.update(e, ids=ids[:W].cpu().numpy(), conf=conf[:W].cpu().numpy())
                e = rec
            self.trace.append(e)
            if P == self.end:
                break
            t += 1
        return self.tok.cpu().numpy()
