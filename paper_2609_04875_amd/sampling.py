"""Deterministic next-token sampling (``pgsr_sample_tokens`` of
``include/pgsr.h``): Gumbel-max over logits / T with Philox4x64-10 noise keyed
by (seed, stream, position), greedy at T = 0.  Marshalling only."""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import numpy as np
import torch

from . import _native as N

_DT = {torch.float32: N.F32, torch.bfloat16: N.BF16}


def sample_workspace_bytes(n: int, vocab: int) -> int:
    return int(N.lib.pgsr_sample_workspace_bytes(n, vocab))


def sample_tokens(logits: torch.Tensor, temperature: float, seed: int, streams: Sequence[int],
                  positions: Sequence[int], out: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Next token per row of ``logits`` [n, vocab] (fp32 or bf16, on the GPU)."""
    assert logits.dim() == 2 and logits.is_contiguous() and logits.dtype in _DT
    n, vocab = logits.shape
    if out is None:
        out = torch.empty(n, dtype=torch.int32, device=logits.device)
    s = np.ascontiguousarray(np.asarray(streams, dtype=np.int64).reshape(n))
    p = np.ascontiguousarray(np.asarray(positions, dtype=np.int64).reshape(n))
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    st = (stream or torch.cuda.current_stream()).cuda_stream
    N.check(N.lib.pgsr_sample_tokens(n, vocab, _DT[logits.dtype], logits.data_ptr(), float(temperature),
                                     ctypes.c_uint64(seed & (2 ** 64 - 1)), s.ctypes.data_as(ctypes.c_void_p),
                                     p.ctypes.data_as(ctypes.c_void_p), ws_ptr, ws_bytes, out.data_ptr(), st))
    return out
