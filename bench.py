"""Benchmark: denoising steps/s of block-wise diffusion-LLM inference on one MI355X.

Workload (default): one LLaDA-8B-shaped denoising step in bf16 with random
N(0, 0.02) weights: 32 layers, d 4096, 32 heads x 128, SwiGLU 12288, vocab
126464; a prefix KV cache of 512 tokens prefilled from random prompt ids; a
32-token block with 24 MASK and 8 committed random ids; each step is
dllm_denoise_step + dllm_commit(k=1), captured once as a HIP graph and replayed
for the timed steps (--eager: plain library calls).  Inputs are synthetic and
resident in HBM before the timed region.

Prints ONE JSON line with the metric, a roofline record for the dominant kernel
(gate/up projection: the largest share of a step's time) and the CPU oracle's
throughput on a bounded sample of the same step.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0

WORKLOADS = {
    # name: (shape, dtype, prefix, window, masked rows, commits per segment, segments)
    "llada8b_bf16_p512_w32": dict(shape="llada8b", dtype="bf16", prefix=512, W=32,
                                  masked=list(range(8, 32)), segs=[(0, 32, 1)]),
    "llada8b_bf16_p1024_w64_spec": dict(shape="llada8b", dtype="bf16", prefix=1024, W=64,
                                        masked=list(range(24, 64)), segs=[(0, 32, 4), (32, 32, 4)], sls=True),
    "llada8b_w8_p4096_w64_spec": dict(shape="llada8b", dtype="w8", prefix=4096, W=64,
                                      masked=list(range(0, 64)), segs=[(0, 32, 2), (32, 32, 2)], sls=True),
    # Q4_0 weights (the paper's own quantisation), otherwise the bf16 step at prefix 512, 32 rows
    "llada8b_q4_p512_w32": dict(shape="llada8b", dtype="q4", prefix=512, W=32,
                                masked=list(range(8, 32)), segs=[(0, 32, 1)]),
    # Dream-7B (grouped-query attention, 28 query heads over 4 K/V heads, Q/K/V biases)
    "dream7b_bf16_p512_w32": dict(shape="dream7b", dtype="bf16", prefix=512, W=32,
                                  masked=list(range(8, 32)), segs=[(0, 32, 1)]),
}
DEFAULT = "llada8b_bf16_p512_w32"
E2E = "llada8b_bf16_e2e128"      # end-to-end 128-token generation (prefill included)
E2E_STAGED = "llada8b_bf16_e2e128_staged"   # the same with staged token stabilisation
E2E_MERGED = "llada8b_bf16_e2e128_merged"   # the same with append + refresh piggybacked on the next step
E2E_MBSD = "llada8b_bf16_e2e128_mbsd"       # the same with multi-block speculative decoding
# prompt processing alone (large M: the GEMMs are MFMA-bound), bf16 and int8 weights
PREFILL = {"llada8b_bf16_prefill512": ("bf16", 512), "llada8b_bf16_prefill4096": ("bf16", 4096),
           "llada8b_w8_prefill4096": ("w8", 4096)}
MFMA_PEAK_TFLOPS = 2500.0        # bf16 dense


def e2e_latency(dl, torch, shape, dev, model, repeats=3):
    """Prompt 512 ids; 4 blocks of 32 decoded left to right, 32 denoising steps per
    block with one commit each; after each block: append it to the prefix and
    refresh 4 seeded positions of it with seeded new ids.  Wall-clock latency of the
    whole generation (prefill included): (best, all) over `repeats` generations after
    one untimed warmup generation."""
    P0, B, S, R = 512, shape.block, 32, 4
    kv = dl.KVCache(model, P0 + 4 * B)
    prompt = torch.from_numpy(synth.prompt_ids(shape, P0)).to(dev)
    picks = [synth.refresh_picks(shape, P0 + b * B, B, R, call=b) for b in range(4)]
    d_picks = [(torch.from_numpy(p).to(dev), torch.from_numpy(n).to(dev)) for p, n in picks]
    tok0, mask0 = synth.window(shape, B, range(B))
    d_tok0, d_mask0 = torch.from_numpy(tok0).to(dev), torch.from_numpy(mask0).to(dev)
    ids = torch.empty(B, dtype=torch.int32, device=dev)
    conf = torch.empty(B, device=dev)
    rid = torch.empty(R, dtype=torch.int32, device=dev)
    rconf = torch.empty(R, device=dev)
    sched = [B // S + (1 if t < B % S else 0) for t in range(S)]

    def generate():
        dl.dllm_prefill(model.handle, kv.handle, prompt, P0)
        for b in range(4):
            tok, mask = d_tok0.clone(), d_mask0.clone()
            for t in range(S):
                dl.dllm_denoise_step(model.handle, kv.handle, tok, mask, B, ids, conf)
                dl.dllm_commit(conf, ids, tok, mask, 0, B, sched[t])
            dl.dllm_append_prefix_kv(model.handle, kv.handle, tok, B)
            p, n = d_picks[b]
            dl.dllm_refresh_kv(model.handle, kv.handle, p, n, R, rid, rconf)
        torch.cuda.synchronize()

    def fresh_kv():
        nonlocal kv
        kv.close()
        kv = dl.KVCache(model, P0 + 4 * B)

    generate()                                  # warmup (untimed)
    times = []
    for _ in range(repeats):
        fresh_kv()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        generate()
        times.append(time.perf_counter() - t0)
    kv.close()
    return min(times), times


def run_e2e(args, dl, torch, shape, dev):
    """End-to-end 128-token generation (e2e_latency) as its own bench line."""
    P0, B, S, R = 512, shape.block, 32, 4
    glob = synth.global_weights(shape, "bf16")
    model = dl.Model(shape, "bf16", glob, lambda l: synth.layer_weights(shape, l, "bf16"), max_window=64,
                     max_pos=P0 + 4 * B + 64)
    lat, times = e2e_latency(dl, torch, shape, dev, model)
    model.close()
    return {
        "metric": "end-to-end 128-token generation latency, LLaDA-8B shape, block 32",
        "value": round(128 / lat, 2), "unit": "tokens/s", "n_gpus": 1, "steps": 128, "warmup": 128,
        "ms_per_step": round(lat * 1000 / 128, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
        "config": {"workload": E2E, "prompt": P0, "blocks": 4, "block": B, "steps_per_block": S,
                   "refresh_per_block": R},
        "latency_s": round(lat, 4), "latencies_s": [round(t, 4) for t in times],
    }


def run_e2e_merged(args, dl, torch, shape, dev):
    """The end-to-end generation of run_e2e with the append and the 4-position
    revision of each completed block piggybacked on the next block's first step
    (dllm_step_merged): the revised ids are written into the completed block, which
    is then appended inside the step's forward (64 rows: 32 appended + 32 window),
    so each block boundary streams the weights once instead of three times.  The
    last block is appended with a merged call without a window."""
    P0, B, S, R = 512, shape.block, 32, 4
    glob = synth.global_weights(shape, "bf16")
    model = dl.Model(shape, "bf16", glob, lambda l: synth.layer_weights(shape, l, "bf16"), max_window=64,
                     max_pos=P0 + 4 * B + 64)
    kv = dl.KVCache(model, P0 + 4 * B + B)
    prompt = torch.from_numpy(synth.prompt_ids(shape, P0)).to(dev)
    picks = [synth.refresh_picks(shape, P0 + b * B, B, R, call=b) for b in range(4)]
    d_picks = [(torch.from_numpy(p - (P0 + b * B)).long().to(dev), torch.from_numpy(n).to(dev))
               for b, (p, n) in enumerate(picks)]
    tok0, mask0 = synth.window(shape, B, range(B))
    d_tok0, d_mask0 = torch.from_numpy(tok0).to(dev), torch.from_numpy(mask0).to(dev)
    ids = torch.empty(B, dtype=torch.int32, device=dev)
    conf = torch.empty(B, device=dev)
    sched = [B // S + (1 if t < B % S else 0) for t in range(S)]

    def generate():
        dl.dllm_prefill(model.handle, kv.handle, prompt, P0)
        done = None                      # the completed block, revised, waiting to be appended
        for b in range(4):
            tok, mask = d_tok0.clone(), d_mask0.clone()
            for t in range(S):
                if t == 0 and done is not None:
                    dl.dllm_step_merged(model.handle, kv.handle, None, None, 0, done, B, tok, mask, B, ids, conf)
                else:
                    dl.dllm_denoise_step(model.handle, kv.handle, tok, mask, B, ids, conf)
                dl.dllm_commit(conf, ids, tok, mask, 0, B, sched[t])
            rel, new = d_picks[b]
            tok[rel] = new                 # revision folded into the block before it is appended
            done = tok
        dl.dllm_step_merged(model.handle, kv.handle, None, None, 0, done, B, None, None, 0)
        torch.cuda.synchronize()

    def fresh_kv():
        nonlocal kv
        kv.close()
        kv = dl.KVCache(model, P0 + 4 * B + B)

    generate()
    times = []
    for _ in range(3):
        fresh_kv()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        generate()
        times.append(time.perf_counter() - t0)
    lat = min(times)
    kv.close()
    model.close()
    return {
        "metric": "end-to-end 128-token generation latency with piggybacked append and revision, LLaDA-8B shape, block 32",
        "value": round(128 / lat, 2), "unit": "tokens/s", "n_gpus": 1, "steps": 128, "warmup": 128,
        "ms_per_step": round(lat * 1000 / 128, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
        "config": {"workload": E2E_MERGED, "prompt": P0, "blocks": 4, "block": B, "steps_per_block": S,
                   "revised_per_block": R},
        "latency_s": round(lat, 4), "latencies_s": [round(t, 4) for t in times],
    }


def run_e2e_staged(args, dl, torch, shape, dev):
    """Prompt 512 ids; 4 blocks of 32 decoded with staged token stabilisation at the
    paper's thresholds (visible 0.7, stable 0.9; the most confident position when
    none passes): each step is dllm_denoise_step + dllm_commit_staged, a block ends
    when no position is invisible, is appended with its visible tokens, and every
    tracked visible prefix token is re-predicted (two refreshes) before the next
    block.  Random N(0, 0.02) weights put every confidence near 1/vocab, so every
    step takes the fallback and every token stays visible: this is the mechanism's
    cost (host sync per step, re-prediction of all visible tokens), not the paper's
    step savings, which need trained weights.  Also times dllm_commit_staged alone."""
    from paper_2606_13740_amd.staged import StagedGenerator

    P0, B, NB = 512, shape.block, 4
    glob = synth.global_weights(shape, "bf16")
    model = dl.Model(shape, "bf16", glob, lambda l: synth.layer_weights(shape, l, "bf16"), max_window=64,
                     max_pos=P0 + NB * B + 64)
    prompt = torch.from_numpy(synth.prompt_ids(shape, P0)).to(dev)
    stats = {}

    def generate():
        kv = dl.KVCache(model, P0 + NB * B)
        dl.dllm_prefill(model.handle, kv.handle, prompt, P0)
        gen = StagedGenerator(model, kv, theta_visible=0.7, theta_stable=0.9)
        refreshed = []
        for _ in range(NB):
            gen.block()
            refreshed.append(len(gen.tracked))
            gen.refresh_visible()
        torch.cuda.synchronize()
        stats.update(steps=list(gen.steps), refreshed=refreshed,
                     fallback_steps=sum(1 for p in gen.promoted if len(p) == 1))
        kv.close()

    generate()                                  # warmup (untimed)
    times = []
    for _ in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        generate()
        times.append(time.perf_counter() - t0)
    lat = min(times)
    # the staged commit kernel alone, 32-position segment
    conf = torch.rand(B, device=dev)
    ids = torch.randint(0, shape.vocab - 1, (B,), dtype=torch.int32, device=dev)
    tok = torch.full((B,), shape.mask_id, dtype=torch.int32, device=dev)
    mask = torch.ones(B, dtype=torch.uint8, device=dev)
    state = torch.zeros(B, dtype=torch.uint8, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n = 200
    e0.record()
    for _ in range(n):
        dl.dllm_commit_staged(conf, ids, tok, mask, state, 0, B, 2.0, 2.0)
    e1.record()
    torch.cuda.synchronize()
    commit_us = e0.elapsed_time(e1) * 1e3 / n
    model.close()
    return {
        "metric": "end-to-end 128-token generation latency with staged token stabilisation, LLaDA-8B shape, block 32",
        "value": round(128 / lat, 2), "unit": "tokens/s", "n_gpus": 1, "steps": sum(stats["steps"]), "warmup": 1,
        "ms_per_step": round(lat * 1000 / sum(stats["steps"]), 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
        "config": {"workload": E2E_STAGED, "prompt": P0, "blocks": NB, "block": B, "theta_visible": 0.7,
                   "theta_stable": 0.9},
        "latency_s": round(lat, 4), "latencies_s": [round(t, 4) for t in times],
        "steps_per_block": stats["steps"], "fallback_steps": stats["fallback_steps"],
        "tracked_visible_before_refresh": stats["refreshed"],
        "commit_staged_us": round(commit_us, 2),
    }


def run_e2e_mbsd(args, dl, torch, shape, dev):
    """Prompt 512 ids; 128 tokens (4 blocks of 32) decoded with multi-block
    speculative decoding: a 32-row window slides along the commit frontier, one
    commit per step, the window grows by the latency table once at most 4 masked
    positions remain in the current block (allowance 10%), draft rows past the
    current block are recorded and accepted when their block becomes current; only
    masked window rows get an LM-head output (selective logits skipping).  The
    latency table is measured first: the window at each row count.  Runs:
    acceptance threshold 0.9 (random weights give confidences near 1e-3, so nothing
    is accepted: the mechanism's cost), 0 (a draft is accepted whenever the current
    step predicts the id it recorded), and 0 with a 15% allowance, which admits the
    48-row window, so lookahead runs at the end of every block."""
    from paper_2606_13740_amd.mbsd import MBSDGenerator

    P0, B, NB, WN = 512, shape.block, 4, 32
    rows = (32, 48, 64)
    glob = synth.global_weights(shape, "bf16")
    model = dl.Model(shape, "bf16", glob, lambda l: synth.layer_weights(shape, l, "bf16"), max_window=max(rows),
                     max_pos=P0 + NB * B + max(rows))
    prompt = torch.from_numpy(synth.prompt_ids(shape, P0)).to(dev)

    # latency table (window rows -> ms per step)
    kv = dl.KVCache(model, P0 + max(rows))
    dl.dllm_prefill(model.handle, kv.handle, prompt, P0)
    tok0, mask0 = synth.window(shape, max(rows), range(max(rows)))
    d_tok, d_mask = torch.from_numpy(tok0).to(dev), torch.from_numpy(mask0).to(dev)
    ids = torch.empty(max(rows), dtype=torch.int32, device=dev)
    conf = torch.empty(max(rows), device=dev)
    # at a lookahead step at most tau = 4 current-block rows and the R - 32 draft rows
    # are masked: the table times the window with that many LM-head rows
    need = torch.zeros(max(rows), dtype=torch.uint8, device=dev)
    need[WN - 4:] = 1
    table = []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for R in rows:
        for _ in range(3):
            dl.dllm_denoise_window_sls(model.handle, kv.handle, P0, d_tok, d_mask, need, R - WN + 4, R, ids, conf)
        e0.record()
        for _ in range(10):
            dl.dllm_denoise_window_sls(model.handle, kv.handle, P0, d_tok, d_mask, need, R - WN + 4, R, ids, conf)
        e1.record()
        torch.cuda.synchronize()
        table.append((R, e0.elapsed_time(e1) / 10))
    kv.close()
    log("latency table " + ", ".join(f"{r}: {t:.3f} ms" for r, t in table))

    def generate(theta, allowance=0.1):
        kv = dl.KVCache(model, P0 + NB * B)
        dl.dllm_prefill(model.handle, kv.handle, prompt, P0)
        gen = MBSDGenerator(model, kv, NB * B, window=WN, k=1, tau=4, latency_table=table, allowance=allowance,
                            theta_accept=theta)
        gen.run()
        torch.cuda.synchronize()
        kv.close()
        tr = gen.trace
        return dict(steps=len(tr), accepted=sum(len(e["accepted"]) for e in tr),
                    lookahead_steps=sum(1 for e in tr if e["R"] > WN), rows_total=sum(e["W"] for e in tr))

    runs = {}
    # (acceptance threshold, lookahead allowance); the last run allows the +12-14% of a
    # 48-row window, so the window grows at the end of every block
    for theta, allowance in ((0.9, 0.1), (0.0, 0.1), (0.0, 0.15)):
        generate(theta, allowance)               # warmup (untimed)
        times = []
        for _ in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            st = generate(theta, allowance)
            times.append(time.perf_counter() - t0)
        key = f"theta {theta}, allowance {allowance}"
        runs[key] = dict(st, latency_s=round(min(times), 4), latencies_s=[round(t, 4) for t in times])
        log(f"mbsd {key}: {runs[key]}")
    model.close()
    main_run = runs["theta 0.9, allowance 0.1"]
    lat = main_run["latency_s"]
    return {
        "metric": "end-to-end 128-token generation latency with multi-block speculative decoding, LLaDA-8B shape, "
                  "block 32",
        "value": round(128 / lat, 2), "unit": "tokens/s", "n_gpus": 1, "steps": main_run["steps"], "warmup": 1,
        "ms_per_step": round(lat * 1000 / main_run["steps"], 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
        "config": {"workload": E2E_MBSD, "prompt": P0, "blocks": NB, "block": B, "window": WN, "commits_per_step": 1,
                   "tau": 4, "allowance": 0.1, "theta_accept": 0.9},
        "latency_table_ms": [[r, round(t, 4)] for r, t in table],
        "runs": runs,
    }


def run_prefill(args, dl, torch, shape, dev):
    """dllm_prefill of a P-token prompt (all layers, no LM head), repeated: prompt
    tokens/s.  The GEMMs multiply P rows, so they are bound by MFMA issue, not by
    HBM: the roofline record reports the gate/up launch's algorithmic flops
    (2 * P * 2F * d, the model's arithmetic; the hi/lo activation planes double the
    MFMAs actually issued) against the bf16 dense MFMA peak.  Per-class durations
    come from events around every launch of the class inside the timed prefills."""
    dtype, P = PREFILL[args.workload]
    glob = synth.global_weights(shape, "bf16")
    t0 = time.time()
    model = dl.Model(shape, dtype, glob, lambda l: synth.layer_weights(shape, l, "bf16"), max_window=64,
                     max_pos=P + 64)
    log(f"model created in {time.time() - t0:.1f} s")
    kv = dl.KVCache(model, P)
    prompt = torch.from_numpy(synth.prompt_ids(shape, P)).to(dev)
    # a prefill needs a cache with prefix_len 0: fresh handles over the same buffer,
    # made before the timed region (a handle is host state only)
    pool = []

    def fresh_handles(n):
        for h in pool:
            dl.dllm_kv_destroy(h)
        pool[:] = [dl.dllm_kv_create(model.handle, kv.buf, kv.nbytes, P) for _ in range(n)]

    def prefill():
        dl.dllm_prefill(model.handle, pool.pop(), prompt, P)

    steps = max(1, min(args.steps, 20 if P <= 512 else 5))
    warm = max(1, min(args.warmup, 2))
    fresh_handles(warm)
    for _ in range(warm):
        prefill()
    torch.cuda.synchronize()
    fresh_handles(steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        prefill()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    log(f"prefill {P}: {ms:.3f} ms")
    d, F, L = shape.d_model, shape.d_ff, shape.n_layers
    dkv = shape.kv_heads * shape.head_dim
    flops = {"qkv": 2.0 * P * (d + 2 * dkv) * d, "oproj": 2.0 * P * d * d, "gateup": 2.0 * P * 2 * F * d,
             "down": 2.0 * P * d * F}
    kern = {}
    for name, cls in dl.KERNEL_CLASSES.items():
        if name == "lmhead":
            continue
        torch.cuda.synchronize()
        fresh_handles(2)
        dl.dllm_probe_enable(model.handle, cls, L * 2)
        for _ in range(2):
            prefill()
        n, probe_ms = dl.dllm_probe_read(model.handle)
        dl.dllm_probe_enable(model.handle, -1, 1)
        rec = {"launches": L, "mean_us": round(probe_ms * 1e3, 2)}
        if name in flops:
            rec["tflops"] = round(flops[name] / (probe_ms * 1e-3) / 1e12, 1)
        kern[name] = rec
    torch.cuda.synchronize()
    fresh_handles(0)
    total_flops = L * sum(flops.values())
    dk = kern["gateup"]
    roof = {"bound": "mfma", "achieved": dk["tflops"], "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(dk["tflops"] / MFMA_PEAK_TFLOPS, 4), "traffic": None, "kernel": "gemm gate/up + SwiGLU",
            "alg_flops_per_launch": flops["gateup"], "mean_launch_us": dk["mean_us"],
            "timing": "HIP events around each gate/up launch inside the prefills"}
    kv.close()
    model.close()
    return {"metric": f"prompt processing (prefill) tokens/sec, LLaDA-8B shape, {P}-token prompt; % of MFMA roofline",
            "value": round(P / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warm,
            "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": {"bf16": "bf16", "w8": "int8w-bf16a"}[dtype],
            "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
            "config": {"workload": args.workload, "layers": L, "d_model": d, "d_ff": F, "prompt": P},
            "gemm_tflops": round(total_flops / (ms * 1e-3) / 1e12, 1), "kernels": kern, "roofline": roof}


def run_sweep(args, dl, torch, shape, dev):
    """Step latency against the window's row count W (prefix 512, bf16): weight
    streaming keeps it nearly flat until the GEMMs become MFMA-bound."""
    P, Ws = 512, [1, 2, 4, 8, 16, 32, 40, 48, 64, 96, 128, 256]
    glob = synth.global_weights(shape, "bf16")
    model = dl.Model(shape, "bf16", glob, lambda l: synth.layer_weights(shape, l, "bf16"), max_window=max(Ws),
                     max_pos=P + max(Ws) + 64)
    kv = dl.KVCache(model, P + max(Ws))
    dl.dllm_prefill(model.handle, kv.handle, torch.from_numpy(synth.prompt_ids(shape, P)).to(dev), P)
    rows = []
    for W in Ws:
        tok, mask = synth.window(shape, W, range(W))
        d_tok, d_mask = torch.from_numpy(tok).to(dev), torch.from_numpy(mask).to(dev)
        ids = torch.empty(W, dtype=torch.int32, device=dev)
        conf = torch.empty(W, device=dev)
        for _ in range(3):
            dl.dllm_denoise_step(model.handle, kv.handle, d_tok, d_mask, W, ids, conf)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 10
        e0.record()
        for _ in range(n):
            dl.dllm_denoise_step(model.handle, kv.handle, d_tok, d_mask, W, ids, conf)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        rows.append({"W": W, "ms_per_step": round(ms, 4), "query_tok_s": round(W * 1000.0 / ms, 1)})
        log(f"W {W}: {ms:.3f} ms")
    kv.close()
    model.close()
    return {"metric": "denoising-step latency against window rows (M-sweep), LLaDA-8B shape, prefix 512",
            "unit": "ms/step", "n_gpus": 1, "higher_is_better": False, "dtype": "bf16",
            "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
            "config": {"workload": "llada8b_bf16_p512_msweep", "prefix": P}, "sweep": rows}


def tiny_times(dl, torch, dev):
    """The tiny fp32 model (2 layers, d 256, vocab 1024): prompt 64 ids prefilled, one
    32-row all-MASK block generated in 4 steps of 8 commits.  Absolute times: one step
    (dllm_denoise_step + dllm_commit, GPU events over 200 steps at the block's first
    step) and one whole generation (prefill + 4 steps, wall clock, best of 20)."""
    sh = synth.TINY
    w = synth.all_weights(sh, "f32", 0)
    model = dl.Model(sh, "f32", {k: w[k] for k in ("embed", "lm_head", "final_norm")}, lambda l: w["layers"][l],
                     max_window=64, max_pos=256)
    prompt = torch.from_numpy(synth.prompt_ids(sh, 64)).to(dev)
    tok0, mask0 = synth.window(sh, 32, range(32))
    d_tok0, d_mask0 = torch.from_numpy(tok0).to(dev), torch.from_numpy(mask0).to(dev)
    ids = torch.empty(32, dtype=torch.int32, device=dev)
    conf = torch.empty(32, device=dev)
    kv = dl.KVCache(model, 96)
    dl.dllm_prefill(model.handle, kv.handle, prompt, 64)
    tok, mask = d_tok0.clone(), d_mask0.clone()
    for _ in range(10):
        dl.dllm_denoise_step(model.handle, kv.handle, d_tok0, d_mask0, 32, ids, conf)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n = 200
    e0.record()
    for _ in range(n):
        dl.dllm_denoise_step(model.handle, kv.handle, d_tok0, d_mask0, 32, ids, conf)
        dl.dllm_commit(conf, ids, tok, mask, 0, 32, 8)
    e1.record()
    torch.cuda.synchronize()
    step_ms = e0.elapsed_time(e1) / n
    kv.close()
    gens = []
    for _ in range(21):
        kv = dl.KVCache(model, 96)
        tok, mask = d_tok0.clone(), d_mask0.clone()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dl.dllm_prefill(model.handle, kv.handle, prompt, 64)
        for _ in range(4):
            dl.dllm_denoise_step(model.handle, kv.handle, tok, mask, 32, ids, conf)
            dl.dllm_commit(conf, ids, tok, mask, 0, 32, 8)
        torch.cuda.synchronize()
        gens.append(time.perf_counter() - t0)
        kv.close()
    model.close()
    return {"workload": "tiny fp32: 2 layers, d 256, prompt 64, one 32-row block in 4 steps of 8 commits",
            "step_ms": round(step_ms, 4), "generation_ms": round(1e3 * min(gens[1:]), 3)}


def measured_read_peak(dl, torch, dev, gib=4):
    """Streaming-read rate of the library's plain read kernel over `gib` GiB (best of 5 launches)."""
    buf = torch.empty(gib << 30, dtype=torch.uint8, device=dev)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    for _ in range(2):
        dl.dllm_read_bandwidth(buf, buf.numel(), sink)
    best = None
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dl.dllm_read_bandwidth(buf, buf.numel(), sink)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1)
        best = t if best is None else min(best, t)
    del buf
    return buf_gbs(gib << 30, best)


def read_floor_us(dl, torch, dev, nbytes, pool):
    """Mean duration of the library's plain streaming read over `nbytes` (the same
    16-byte non-temporal loads the GEMMs use), launched back to back over consecutive
    windows of a >= 2 GiB pool (so the 256 MB Infinity Cache cannot serve them): the
    floor a kernel that only reads that many bytes reaches, its launch included."""
    n16 = (int(nbytes) + 15) // 16 * 16
    nwin = max(1, pool.numel() // n16)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    base = pool.data_ptr()
    for i in range(4):
        dl.lib().dllm_read_bandwidth(base + (i % nwin) * n16, n16, sink.data_ptr(), None)
    n = 32
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(n):
        dl.lib().dllm_read_bandwidth(base + (i % nwin) * n16, n16, sink.data_ptr(), None)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / n


def buf_gbs(nbytes, ms):
    return nbytes / (ms * 1e-3) / 1e9


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# The dominant kernel's measured HBM bytes come from the committed rocprofv3 counter
# summary of this workload (FETCH_SIZE / WRITE_SIZE scaled by a 1 GiB copy).
COUNTERS = os.path.join(ROOT, "profiles", "hbm_counters_llada8b_bf16_p512_w32.txt")
DOMINANT = "gemm_kernel<1, 6, 1, 8, 2, dllm::EpiSwiGLU<false> >"


def measured_traffic(workload):
    if workload != DEFAULT or not os.path.exists(COUNTERS):
        return None
    for line in open(COUNTERS):
        if DOMINANT in line:
            parts = line.split()
            try:
                return round((float(parts[-2]) + float(parts[-1])) * 1e6)
            except ValueError:
                return None
    return None


def cpu_baseline(shape, dtype, wl, prompt, tok, mask, glob, min_s=10.0):
    """Oracle (float64 NumPy) on a bounded sample of the same step: whole steps whose
    layer forward runs n_layers times on one layer's weights (every layer has the
    same shapes, so the same arithmetic and memory traffic), then the final norm,
    the LM head and the confidences; repeated until at least min_s seconds."""
    import oracle

    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    sh1 = shape.with_layers(1)
    om = oracle.OracleModel(sh1, dict(glob, layers=None), int8=(dtype == "w8"), q4=(dtype == "q4"), cache_layers=True,
                            layer_source=lambda l: synth.layer_weights(shape, l, "bf16"))
    kv = oracle.OracleKV(sh1, wl["prefix"] + wl["W"])
    oracle.prefill(om, kv, prompt)        # setup, not timed
    P, W = wl["prefix"], wl["W"]
    ids = oracle.input_ids(shape, tok, mask)
    steps, t_layers, t_head = 0, 0.0, 0.0
    while t_layers + t_head < min_s:
        t0 = time.perf_counter()
        for _ in range(shape.n_layers):
            x, _ = oracle.forward_rows(om, kv, ids, P + np.arange(W), np.full(W, P + W), lm_head=False)
        t1 = time.perf_counter()
        logits = om.lm_logits(oracle.rmsnorm(x, om.final_norm, shape.eps))
        oracle.confidence(logits)
        t2 = time.perf_counter()
        steps, t_layers, t_head = steps + 1, t_layers + (t1 - t0), t_head + (t2 - t1)
    return {"value": steps / (t_layers + t_head), "unit": "steps/s", "cores": cores, "kind": "oracle",
            "sample": f"{steps} whole steps ({t_layers + t_head:.1f} s): the layer forward {shape.n_layers}x per "
                      f"step on layer 0's weights ({t_layers / steps:.2f} s per step) + the full LM head and "
                      f"confidences ({t_head / steps:.2f} s per step); float64 NumPy"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT,
                    choices=sorted(WORKLOADS) + [E2E, E2E_STAGED, E2E_MERGED, E2E_MBSD] + sorted(PREFILL))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="default workload: skip the end-to-end, tiny-model, M-sweep and read-floor measurements "
                         "(short runs under a counter profiler)")
    ap.add_argument("--eager", action="store_true",
                    help="time plain library calls instead of replays of the step captured as a HIP graph")
    ap.add_argument("--no-sls", action="store_true",
                    help="run the LM head over every window row (no selective logits skipping)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (3 launches): the reference for HBM byte counters")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the metric: step latency against the window's row count (M-sweep)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel() * 4, "launches": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the path has no multi-GPU mode",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2606_13740_amd as dl

    if args.workload in (E2E, E2E_STAGED, E2E_MERGED, E2E_MBSD):
        torch.cuda.set_device(0)
        run = {E2E: run_e2e, E2E_STAGED: run_e2e_staged, E2E_MERGED: run_e2e_merged,
               E2E_MBSD: run_e2e_mbsd}[args.workload]
        print(json.dumps(run(args, dl, torch, synth.LLADA_8B, torch.device("cuda:0"))), flush=True)
        return
    if args.workload in PREFILL:
        torch.cuda.set_device(0)
        print(json.dumps(run_prefill(args, dl, torch, synth.LLADA_8B, torch.device("cuda:0"))), flush=True)
        return
    if args.sweep:
        torch.cuda.set_device(0)
        print(json.dumps(run_sweep(args, dl, torch, synth.LLADA_8B, torch.device("cuda:0"))), flush=True)
        return
    wl = WORKLOADS[args.workload]
    shape = synth.PRESETS[wl["shape"]]
    dtype = wl["dtype"]
    P, W = wl["prefix"], wl["W"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t0 = time.time()
    glob = synth.global_weights(shape, "bf16")
    # the default workload's model also serves the end-to-end generation (prompt 512 +
    # 128 tokens) and the down-projection M-sweep (windows up to 256 rows)
    extras = args.workload == DEFAULT and not args.no_extras
    model = dl.Model(shape, dtype, glob, lambda l: synth.layer_weights(shape, l, "bf16"),
                     max_window=256 if extras else 64, max_pos=max(P + W + 64, 1024 if extras else 0))
    log(f"model created in {time.time() - t0:.1f} s")
    kv = dl.KVCache(model, P + W)
    prompt = synth.prompt_ids(shape, P)
    dl.dllm_prefill(model.handle, kv.handle, torch.from_numpy(prompt).to(dev), P)
    tok, mask = synth.window(shape, W, wl["masked"])
    d_tok0 = torch.from_numpy(tok).to(dev)
    d_mask0 = torch.from_numpy(mask).to(dev)
    d_tok, d_mask = d_tok0.clone(), d_mask0.clone()
    ids = torch.empty(W, dtype=torch.int32, device=dev)
    conf = torch.empty(W, device=dev)
    cpos = torch.empty(64, dtype=torch.int32, device=dev)
    ncom = torch.empty(4, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    log(f"prefill {P} done")

    # selective logits skipping: only masked rows need an LM-head output; the bound is
    # the masked count at the start (commits only shrink the set)
    sls = wl.get("sls", False) and not args.no_sls
    n_need = len(wl["masked"])

    def step():
        if sls:
            dl.dllm_denoise_window_sls(model.handle, kv.handle, P, d_tok, d_mask, d_mask, n_need, W, ids, conf)
        else:
            dl.dllm_denoise_step(model.handle, kv.handle, d_tok, d_mask, W, ids, conf)
        for j, (b, n, k) in enumerate(wl["segs"]):
            dl.dllm_commit(conf, ids, d_tok, d_mask, b, n, k, cpos[16 * j:], ncom[j:])

    # The timed steps replay the step (its launches and the commits) captured once as a
    # HIP graph: the same kernels with the same arguments, without the host's
    # per-launch work (--eager: plain calls).
    run = step
    if not args.eager:
        from paper_2606_13740_amd.graph import StepGraph

        run = StepGraph(step).replay
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    d_tok.copy_(d_tok0)
    d_mask.copy_(d_mask0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = e0.elapsed_time(e1) / args.steps
    steps_s = 1000.0 / ms
    commits = sum(k for _, _, k in wl["segs"])
    log(f"{ms:.3f} ms/step (GPU events), wall {1000 * wall / args.steps:.3f} ms/step")

    # Per-kernel durations, after the timed region, on the launch stream:
    #  - replay: the step's own launches of one kernel class (same kernels, launch
    #    shapes and operands), layer after layer back to back between two events;
    #    mean = elapsed / launches (dllm_kernel_replay);
    #  - probe: events around every launch of the class inside real steps, which adds
    #    the event records' own latency to each launch.
    kern = {}
    step_bytes = 0.0
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for name, cls in dl.KERNEL_CLASSES.items():
        nl = 1 if name == "lmhead" else shape.n_layers
        dl.dllm_probe_enable(model.handle, cls, nl * 4)
        for _ in range(4):
            step()
        n, probe_ms = dl.dllm_probe_read(model.handle)
        dl.dllm_probe_enable(model.handle, -1, 1)
        n_rep = 2 * shape.n_layers if name != "lmhead" else 16
        dl.dllm_kernel_replay(model.handle, kv.handle, cls, W, n_rep)       # warm
        r0.record()
        dl.dllm_kernel_replay(model.handle, kv.handle, cls, W, n_rep)
        r1.record()
        torch.cuda.synchronize()
        mean_ms = r0.elapsed_time(r1) / n_rep
        b = dl.dllm_kernel_bytes(model.handle, cls, W, P)
        kern[name] = {"launches_per_step": nl, "mean_us": mean_ms * 1e3, "probe_us": probe_ms * 1e3, "alg_bytes": b,
                      "gbs": b / (mean_ms * 1e-3) / 1e9 if mean_ms > 0 else None}
        step_bytes += nl * b
    step()                          # leave the workspaces as a step leaves them
    torch.cuda.synchronize()
    read_gbs = measured_read_peak(dl, torch, dev)
    # per-size floor: a plain read of each class's algorithmic bytes
    pool = None
    if not args.no_extras:
        pool = torch.empty(max(2 << 30, int(4.2 * max(v["alg_bytes"] for v in kern.values()))), dtype=torch.uint8,
                           device=dev)
    for name, v in kern.items():
        if pool is None:
            break
        f = read_floor_us(dl, torch, dev, v["alg_bytes"], pool)
        v["read_floor_us"] = f
        v["frac_of_read_floor"] = f / v["mean_us"] if v["mean_us"] > 0 else None
    del pool
    dom = "gateup"
    dk = kern[dom]
    traffic = measured_traffic(args.workload)
    roof = {"bound": "hbm", "achieved": round(dk["gbs"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dk["gbs"] / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": "gemm gate/up + SwiGLU",
            "alg_bytes_per_launch": dk["alg_bytes"], "mean_launch_us": round(dk["mean_us"], 2),
            "timing": "the step's gate/up launches replayed back to back, layer by layer (HIP events)",
            "measured_read_peak": round(read_gbs, 1), "frac_of_measured": round(dk["gbs"] / read_gbs, 4)}

    out = {
        "metric": ("denoising steps/sec + tokens/sec, LLaDA-8B shape, block 32; % of HBM roofline"
                   if wl["shape"] == "llada8b" else
                   "denoising steps/sec + tokens/sec, Dream-7B shape, block 32; % of HBM roofline"),
        "value": round(steps_s, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "w8": "int8w-bf16a", "q4": "q4_0w-bf16a"}[dtype],
        "data": "synthetic (seeded N(0,0.02) weights, uniform ids)",
        "config": {"workload": args.workload, "layers": shape.n_layers, "d_model": shape.d_model,
                   "heads": shape.n_heads, "kv_heads": shape.kv_heads, "head_dim": shape.head_dim,
                   "d_ff": shape.d_ff, "vocab": shape.vocab,
                   "prefix": P, "window": W, "masked": len(wl["masked"]), "commits_per_step": commits,
                   "lm_head_rows": n_need if sls else W},
        "launch": "eager library calls" if args.eager else "HIP graph replay of the step + commits",
        "query_tok_s": round(W * steps_s, 1),
        "committed_tok_s": round(commits * steps_s, 1),
        "step_hbm_frac": round(step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "step_hbm_frac_of_measured": round(step_bytes / (ms * 1e-3) / 1e9 / read_gbs, 4),
        "step_alg_gb": round(step_bytes / 1e9, 3),
        "kernels": {k: {kk: (round(vv, 2) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kern.items()},
        "roofline": roof,
    }
    # the dispatch gap: step time minus the per-class replay time of its launches (the
    # replays include each launch's own ramp and drain; the gap holds the embedding, the
    # LM-head merge, the commit and the switches between kernels)
    class_ms = sum(v["launches_per_step"] * v["mean_us"] for v in kern.values()) / 1e3
    out["dispatch_gap_ms"] = round(ms - class_ms, 4)
    out["sum_of_class_replays_ms"] = round(class_ms, 4)
    if extras:
        # down projection alone (GEMM + its residual reduction) against the window's rows:
        # latency stays flat while the weight stream dominates
        kv_s = dl.KVCache(model, 256)
        sweep = []
        for Ws in (1, 2, 4, 8, 16, 32, 64, 128, 256):
            dl.dllm_kernel_replay(model.handle, kv_s.handle, dl.K_DOWN, Ws, shape.n_layers)
            r0.record()
            dl.dllm_kernel_replay(model.handle, kv_s.handle, dl.K_DOWN, Ws, 2 * shape.n_layers)
            r1.record()
            torch.cuda.synchronize()
            sweep.append([Ws, round(r0.elapsed_time(r1) * 1e3 / (2 * shape.n_layers), 2)])
        kv_s.close()
        out["down_proj_msweep_us"] = sweep
        lat, lats = e2e_latency(dl, torch, shape, dev, model, repeats=2)
        out["e2e128"] = {"workload": "llada8b_bf16_e2e128: prompt 512, 4 blocks x 32 steps (1 commit each), "
                                     "append + 4-row refresh per block", "latency_s": round(lat, 4),
                         "tokens_s": round(128 / lat, 2), "latencies_s": [round(t, 4) for t in lats]}
        out["tiny_fp32"] = tiny_times(dl, torch, dev)
        log(f"e2e {lat:.3f} s; tiny {out['tiny_fp32']}")
    if not args.no_cpu_baseline:
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(shape, dtype, wl, prompt, tok, mask, glob)
        log(f"cpu baseline in {time.time() - t0:.1f} s")
    kv.close()
    model.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
