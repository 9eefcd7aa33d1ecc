"""Oracle for the block-wise diffusion-LLM denoising step (float64 NumPy).

TEST INFRASTRUCTURE: imported only by the tests, the smoke check and the
benchmark's CPU-baseline leg.  The product path never imports it.
"""
from .model import (  # noqa: F401
    IV, S, V, OracleKV, OracleModel, StepOut, append_block, attend, attend_masked, block_causal_allowed,
    commit, commit_schedule, commit_staged, confidence, denoise_step, denoise_window, denoise_window_sls,
    dequantize_q4_0, dequantize_rows, forward_full,
    forward_rows, input_ids, prefill, quantize_rows_int8, quantize_rows_q4_0, refresh, repredict_tracked, rmsnorm, rope,
    silu, skip_logits, softmax,
)
from . import mbsd  # noqa: F401,E402
