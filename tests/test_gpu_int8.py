"""int8 weights on the GPU: the quantiser, code for code, against the oracle.

dllm_quantize_int8 runs the quantiser dllm_model_create applies to DLLM_W8 models
(the same device functions): per output row, in fp32, s = max|w| / 127 and
q = round-half-even(w / s) clamped to [-127, 127], both divisions correctly rounded.
The oracle's quantiser is pinned on the CPU against exact rational arithmetic
(tests/test_oracle.py), so the GPU's codes and scales must equal it bit for bit:
on random bf16 matrices at the LLaDA-8B widths (ragged row counts), on fp32 rows
whose quotients sit exactly halfway between integers, and on fp32 rows whose
float32 quotient rounds to a different integer than the exact one.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2606_13740_amd as dl  # noqa: E402


def _quantize_gpu(w):
    rows, K = w.shape
    if w.dtype == np.uint16:
        src, code = torch.from_numpy(w.view(np.int16)).cuda(), dl.DLLM_BF16
    else:
        src, code = torch.from_numpy(np.ascontiguousarray(w, np.float32)).cuda(), dl.DLLM_F32
    q = torch.full((rows, K), 99, dtype=torch.int8, device="cuda")
    s = torch.full((rows,), -1.0, dtype=torch.float32, device="cuda")
    dl.dllm_quantize_int8(src, code, rows, K, q, s)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


def _check(w):
    q, s = _quantize_gpu(w)
    qo, so = oracle.quantize_rows_int8(synth.as_f32(w) if w.dtype == np.uint16 else w)
    np.testing.assert_array_equal(s.view(np.uint32), so.view(np.uint32))
    bad = np.argwhere(q != qo)
    assert len(bad) == 0, f"{len(bad)} codes differ, first at {bad[:5].tolist()}"


@pytest.mark.parametrize("shape,name,rows", [("llada8b", "wq", 4096), ("llada8b", "wg", 1000),
                                              ("llada8b", "wd", 37), ("small", "wd", 3)])
def test_int8_codes_bit_exact_on_bf16_weights(shape, name, rows):
    sh = synth.LLADA_8B if shape == "llada8b" else synth.SMALL_BF16     # small wd: K = 688, a ragged width
    w = np.ascontiguousarray(synth.weight(sh, name, 0, "bf16")[:rows])
    print(f"case: int8 quantiser, bf16 {w.shape[0]} x {w.shape[1]}", flush=True)
    w[min(1, rows - 1)] = 0                                   # a zero row: s = 0, codes 0
    _check(w)


def _boundary_rows(seed):
    """fp32 rows: element 0 is the row's maximum, the others sit within a few float32
    ulps of (k + 1/2) * s for random k, s = float32(max / 127), so that the quotient's
    float32 rounding decides the code."""
    rng = np.random.default_rng(seed)
    rows = []
    for _ in range(64):
        amax = np.float32(rng.uniform(0.01, 0.1))
        s32 = np.float32(amax / np.float32(127))
        row = [amax if rng.random() < 0.5 else -amax]
        for k in rng.integers(-120, 120, 255):
            w = np.float32((k + 0.5) * float(s32))
            for _ in range(int(rng.integers(0, 4))):
                w = np.nextafter(w, np.float32(np.inf if rng.random() < 0.5 else -np.inf), dtype=np.float32)
            row.append(w)
        rows.append(row)
    return np.array(rows, np.float32)


def test_int8_codes_bit_exact_at_rounding_boundaries():
    print("case: int8 quantiser, halfway and near-halfway fp32 rows", flush=True)
    halfway = np.array([[127.0, 0.5, 1.5, 2.5, -0.5, -2.5, 3.5, -126.5]], np.float32)
    q, s = _quantize_gpu(halfway)
    assert s[0] == np.float32(1.0) and q[0].tolist() == [127, 0, 2, 2, 0, -2, 4, -126]
    for seed in range(4):
        _check(_boundary_rows(seed))
