"""The no-allocation step (dllm_denoise_step_noalloc) through the C ABI against
dllm_denoise_step, the entry point it is a variant of.

Both run the same kernels; only the scratch differs (the library's static device
array instead of the model's workspace), so ids and confidences must be identical.
Two calls in a row, the second with a smaller window, check that nothing of the
first call's scratch leaks into the second; a bf16 case at the LLaDA-8B widths
checks the size that the benchmark's step takes, and a model whose step needs
more than the static array is rejected before any launch.
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


def _both(model, kv, tok, mask):
    W = len(tok)
    out = []
    for f in (dl.dllm_denoise_step, dl.dllm_denoise_step_noalloc):
        ids = torch.full((W,), -7, dtype=torch.int32, device="cuda")
        conf = torch.full((W,), -1.0, device="cuda")
        f(model.handle, kv.handle, dev_i32(tok), dev_u8(mask), W, ids, conf)
        torch.cuda.synchronize()
        out.append((ids.cpu().numpy(), conf.cpu().numpy()))
    return out


def _check_pair(model, kv, W, masked):
    tok, mask = synth.window(model.shape, W, masked)
    (i0, c0), (i1, c1) = _both(model, kv, tok, mask)
    print(f"  W {W}: {int(np.sum(i0 == i1))}/{W} ids equal", flush=True)
    np.testing.assert_array_equal(i1, i0)
    np.testing.assert_array_equal(c1, c0)
    assert np.all(c1 > 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "w8"])
def test_noalloc_step_equals_step_two_calls_shrinking(dtype):
    sh = synth.TINY if dtype == "f32" else synth.SMALL_BF16
    print(f"case: no-alloc step, {dtype}", flush=True)
    model, _, _ = build_pair(sh, dtype, max_window=64, max_pos=512, oracle_too=False)
    kv = dl.KVCache(model, 64 + 64)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(sh, 64)), 64)
    _check_pair(model, kv, 64, list(range(8, 64)))
    _check_pair(model, kv, 17, list(range(3, 17)))
    kv.close()
    model.close()


def test_noalloc_step_8b_width():
    sh = synth.LLADA_8B.with_layers(2)
    print("case: no-alloc step, LLaDA-8B widths, 2 layers, prefix 512", flush=True)
    glob = synth.global_weights(sh, "bf16")
    layers = [synth.layer_weights(sh, l, "bf16") for l in range(sh.n_layers)]
    model = dl.Model(sh, "bf16", glob, lambda l: layers[l], max_window=64, max_pos=640)
    kv = dl.KVCache(model, 512 + 64)
    dl.dllm_prefill(model.handle, kv.handle, dev_i32(synth.prompt_ids(sh, 512)), 512)
    _check_pair(model, kv, 64, list(range(24, 64)))
    _check_pair(model, kv, 32, list(range(8, 32)))
    kv.close()
    model.close()


def test_noalloc_step_rejects_a_step_beyond_the_scratch():
    """A 256-row window at the LLaDA-8B widths needs more than the static 64 MiB: the
    call fails with E_CAPACITY before any launch and the model keeps working."""
    sh = synth.LLADA_8B.with_layers(1)
    glob = synth.global_weights(sh, "bf16")
    lw = synth.layer_weights(sh, 0, "bf16")
    model = dl.Model(sh, "bf16", glob, lambda l: lw, max_window=256, max_pos=512)
    kv = dl.KVCache(model, 256)
    tok, mask = synth.window(sh, 256, range(256))
    ids = torch.empty(256, dtype=torch.int32, device="cuda")
    conf = torch.empty(256, device="cuda")
    with pytest.raises(dl.DllmError) as e:
        dl.dllm_denoise_step_noalloc(model.handle, kv.handle, dev_i32(tok), dev_u8(mask), 256, ids, conf)
    assert e.value.code == dl.DLLM_E_CAPACITY
    dl.dllm_denoise_step(model.handle, kv.handle, dev_i32(tok[:8]), dev_u8(mask[:8]), 8, ids, conf)
    torch.cuda.synchronize()
    kv.close()
    model.close()
