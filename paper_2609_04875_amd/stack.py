"""Stacked-layer replay: F of Eq. (1) as several random-init attention layers.

The paper defines no layer; the stacked workload reads F per layer as
Q = X Wq, K = X Wk, V = X Wv, O = attention(Q, [K_cache; K], [V_cache; V]),
X <- X + O Wo (bf16 storage between steps, no norm, MLP or RoPE).  Every step
is a library call: three projections and the output projection with its
residual on the MFMA GEMM, the attention through the paged pool (one pool
layer per model layer, one shared block table).  Blocks are reserved by the
first layer's replay and the lengths advance (COMMIT) on the last.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import _native as N
from .pool import KVPool, gemm_bf16


class StackedReplay:
    def __init__(self, weights: Sequence[Sequence[torch.Tensor]], n_q_heads: int, n_kv_heads: int,
                 head_dim: int, n_blocks: int, max_seqs: int, max_blocks_per_seq: int,
                 block_size: int = 16, workspace_bytes: int = 0):
        """``weights``: per layer (Wq [Hq*d, dm], Wk [Hkv*d, dm], Wv [Hkv*d, dm],
        Wo [dm, Hq*d]) as bf16 CUDA tensors in the linear-layer [out][in] layout."""
        self.w = [tuple(layer) for layer in weights]
        self.hq, self.hkv, self.d = n_q_heads, n_kv_heads, head_dim
        self.d_model = self.w[0][0].shape[1]
        self.pool = KVPool(len(self.w), n_q_heads, n_kv_heads, head_dim, n_blocks, max_seqs,
                           max_blocks_per_seq, N.BF16, block_size, workspace_bytes=workspace_bytes)
        self._buf = {}

    def _scratch(self, name: str, shape) -> torch.Tensor:
        t = self._buf.get(name)
        if t is None or t.numel() < int(torch.tensor(shape).prod()):
            t = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
            self._buf[name] = t
        return t.view(-1)[: int(torch.tensor(shape).prod())].view(shape)

    def _run(self, fn, seq: int, x: torch.Tensor, scale: float,
             record: Optional[list] = None) -> torch.Tensor:
        """Push the token states x [n, dm] through every layer; returns the new x.
        ``record`` (a list) receives a copy of each layer's attention output."""
        n = x.shape[0]
        q = self._scratch("q", (n, self.hq * self.d))
        k = self._scratch("k", (n, self.hkv * self.d))
        v = self._scratch("v", (n, self.hkv * self.d))
        o = self._scratch("o", (n, self.hq * self.d))
        x = x.clone()
        last = len(self.w) - 1
        for li, (wq, wk, wv, wo) in enumerate(self.w):
            gemm_bf16(x, wq, out=q)
            gemm_bf16(x, wk, out=k)
            gemm_bf16(x, wv, out=v)
            rc = fn(li, [seq], [n], q, k, v, o, scale, commit=(li == last))
            if rc:
                raise N.PgsrError(rc, N.lib.pgsr_last_error().decode())
            if record is not None:
                record.append(o.clone())
            gemm_bf16(o, wo, r=x, out=x)               # x <- x + O Wo
        return x

    def replay(self, seq: int, x: torch.Tensor, scale: float, record: Optional[list] = None) -> torch.Tensor:
        """Replay tokens at positions len(seq) .. len(seq)+n-1 (Algorithm 1, replay loop)."""
        return self._run(self.pool.replay, seq, x, scale, record)

    def full_reset(self, seq: int, x: torch.Tensor, scale: float, record: Optional[list] = None) -> torch.Tensor:
        """Baseline B5: crop to 0 (on the first layer) and replay all of x."""
        return self._run(self.pool.full_reset, seq, x, scale, record)

    def crop(self, seqs: List[int], new_lens: List[int]) -> int:
        return self.pool.crop(seqs, new_lens)
