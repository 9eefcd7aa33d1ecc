"""Steps replayed from a captured HIP graph (paper_2606_13740_amd.graph.StepGraph)
against the same steps run eagerly: the 32-row step + commit, and the 64-row speculative
window step with selective logits + per-segment commits (bf16 and int8 weights, and the
int8 workload's 8B-width launch at prefix 4096 with its 15-split attention).

A replay launches exactly the captured kernels, so every replay must be
bit-identical to the eager call from the same state.  Each test replays several
times with the program's own eager work and synchronisations in between (an eager
step into other buffers, torch arithmetic), and checks every replay.
"""
import numpy as np
import pytest

import synth
from gpu_util import build_pair, dev_i32, dev_u8

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402
from paper_2606_13740_amd.graph import StepGraph  # noqa: E402


def _setup(shape, dtype, P, W, masked):
    model, _, _ = build_pair(shape, dtype, max_pos=P + W + 64, oracle_too=False)
    kv = dl.KVCache(model, P + W)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(shape, P)), P)
    tok, mask = synth.window(shape, W, masked)
    return model, kv, tok, mask


def _other_eager_work(model, kv, tok, mask):
    """An eager step into its own buffers and some torch arithmetic, synchronised."""
    W = len(tok)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    dl.dllm_denoise_step(model.handle, kv.handle, dev_i32(tok), dev_u8(mask), W, ids, conf)
    x = torch.randn(1 << 16, device="cuda")
    _ = (x * 2 + 1).sum()
    torch.cuda.synchronize()


@pytest.mark.parametrize("shape,dtype", [(synth.SMALL_BF16, "bf16"), (synth.TINY, "f32")])
def test_step_and_commit_replays_equal_eager_steps(shape, dtype):
    P, W, n = 96, 32, 8
    print(f"case: graph of step + commit, {dtype}, prefix {P}, window {W}, {n} replays", flush=True)
    model, kv, tok, mask = _setup(shape, dtype, P, W, range(W))
    d_tok0, d_mask0 = dev_i32(tok), dev_u8(mask)
    d_tok, d_mask = d_tok0.clone(), d_mask0.clone()
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    cpos = torch.empty(16, dtype=torch.int32, device="cuda")
    ncom = torch.empty(1, dtype=torch.int32, device="cuda")

    def step():
        dl.dllm_denoise_step(model.handle, kv.handle, d_tok, d_mask, W, ids, conf)
        dl.dllm_commit(conf, ids, d_tok, d_mask, 0, W, 2, cpos, ncom)

    def reset():
        d_tok.copy_(d_tok0)
        d_mask.copy_(d_mask0)
        torch.cuda.synchronize()

    def snapshot():
        return [t.cpu().numpy().copy() for t in (ids, conf, d_tok, d_mask, cpos[:2], ncom)]

    eager = []
    for _ in range(n):
        step()
        torch.cuda.synchronize()
        eager.append(snapshot())
    reset()
    g = StepGraph(step)
    reset()
    for i in range(n):
        ids.fill_(-7)
        conf.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        got = snapshot()
        for a, b in zip(got, eager[i]):
            np.testing.assert_array_equal(a, b)
        _other_eager_work(model, kv, tok, mask)
    assert int(d_mask.sum()) == W - 2 * n                               # the commits really happened
    kv.close()
    model.close()


def test_step_graph_at_8b_width_equals_eager():
    """The benchmark's launch configuration (8B widths, 32-row window, prefix 512; 2 layers)."""
    sh = synth.LLADA_8B.with_layers(2)
    P, W = 512, 32
    print(f"case: graph of the step at 8B width, prefix {P}, window {W}", flush=True)
    model, kv, tok, mask = _setup(sh, "bf16", P, W, range(8, 32))
    d_tok, d_mask = dev_i32(tok), dev_u8(mask)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")

    def step():
        dl.dllm_denoise_step(model.handle, kv.handle, d_tok, d_mask, W, ids, conf)

    step()
    torch.cuda.synchronize()
    ref = (ids.cpu().numpy().copy(), conf.cpu().numpy().copy())
    g = StepGraph(step)
    for _ in range(4):
        ids.fill_(-7)
        conf.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(ids.cpu().numpy(), ref[0])
        np.testing.assert_array_equal(conf.cpu().numpy(), ref[1])
        _other_eager_work(model, kv, tok, mask)
    kv.close()
    model.close()


def _spec_step_graph(shape, dtype, P, W, masked, segs, n):
    """The speculative window step as the 64-row workloads run it: dllm_denoise_window_sls over
    the masked rows (LM head over at most n_need of them) and one dllm_commit per segment,
    replayed n times against the same sequence run eagerly from the same state."""
    model, kv, tok, mask = _setup(shape, dtype, P, W, masked)
    d_tok0, d_mask0 = dev_i32(tok), dev_u8(mask)
    d_tok, d_mask = d_tok0.clone(), d_mask0.clone()
    n_need = len(masked)
    ids = torch.empty(W, dtype=torch.int32, device="cuda")
    conf = torch.empty(W, device="cuda")
    cpos = torch.empty(16 * len(segs), dtype=torch.int32, device="cuda")
    ncom = torch.empty(len(segs), dtype=torch.int32, device="cuda")

    def step():
        dl.dllm_denoise_window_sls(model.handle, kv.handle, P, d_tok, d_mask, d_mask, n_need, W, ids, conf)
        for j, (b, ln, k) in enumerate(segs):
            dl.dllm_commit(conf, ids, d_tok, d_mask, b, ln, k, cpos[16 * j:], ncom[j:])

    def reset():
        d_tok.copy_(d_tok0)
        d_mask.copy_(d_mask0)
        torch.cuda.synchronize()

    def snapshot():
        return [t.cpu().numpy().copy() for t in (ids, conf, d_tok, d_mask, ncom)]

    eager = []
    for _ in range(n):
        step()
        torch.cuda.synchronize()
        eager.append(snapshot())
    reset()
    g = StepGraph(step)
    reset()
    for i in range(n):
        ids.fill_(-7)
        conf.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(snapshot(), eager[i]):
            np.testing.assert_array_equal(a, b)
        _other_eager_work(model, kv, tok, mask)
    committed = sum(k for _, _, k in segs) * n
    assert int(d_mask.sum()) == len(masked) - committed           # the commits really happened
    kv.close()
    model.close()


@pytest.mark.parametrize("dtype", ["bf16", "w8"])
def test_spec_window_step_replays_equal_eager_steps(dtype):
    print(f"case: graph of the 64-row SLS step + 2 segment commits, {dtype}, prefix 160", flush=True)
    _spec_step_graph(synth.SMALL_BF16, dtype, 160, 64, list(range(8, 64)), [(0, 32, 2), (32, 32, 2)], 6)


def test_spec_window_step_graph_at_8b_width_int8_prefix_4096():
    """The int8 64-row workload's launch configuration (8B widths, prefix 4096: the 15-split
    attention and its merge; 2 layers)."""
    print("case: graph of the int8 64-row SLS step at 8B width, prefix 4096", flush=True)
    _spec_step_graph(synth.LLADA_8B.with_layers(2), "w8", 4096, 64, list(range(0, 64)), [(0, 32, 2), (32, 32, 2)], 3)
