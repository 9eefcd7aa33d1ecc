"""Steps replayed from a captured HIP graph (paper_2606_13740_amd.graph.StepGraph)
against the same steps run eagerly.

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
