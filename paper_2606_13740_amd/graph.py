"""Replaying a fixed sequence of library calls from a captured HIP graph.

A denoising step over fixed buffers (the same model, cache, window buffers and
prefix length) launches the same kernels with the same arguments every time and,
once the model's workspace has grown to the window, makes no host synchronisation,
allocation or memset: such a sequence (for example dllm_denoise_step followed by
dllm_commit) can be captured once on a stream and replayed, which takes the host's
per-launch work off every later step.

A capture fixes every pointer and size passed and the cache's prefix length at the
time of capture: capture again after an append, a refresh, or for another window
size.  Calls that copy to the host (dllm_refresh_kv, dllm_step_merged with refresh
rows, dllm_probe_read) or record probe events cannot be captured.

This module only drives torch's graph capture around library calls on the current
stream; every launch in the graph is the library's own.
"""
from typing import Callable


class StepGraph:
    """Captures the launches `fn` makes on the current stream.

    `fn` runs `warmup` times first, eagerly on a side stream (so that any workspace
    growth and its allocation happen before the capture), then once under capture,
    which records its launches without running them.  The eager runs' side effects
    (commits, cache rows) are the caller's to undo before the first replay().
    """

    def __init__(self, fn: Callable[[], None], warmup: int = 2):
        import torch

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(warmup):
                fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            fn()
        torch.cuda.synchronize()

    def replay(self) -> None:
        """Launches the captured sequence on the current stream."""
        self.graph.replay()
