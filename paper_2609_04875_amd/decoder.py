"""Full decoder-layer replay: F of Eq. (1) at the real geometries.

Per layer (pre-norm, as in the public architecture of the model families the
paper runs): h = RMSNorm(x) g_attn; Q, K, V = h Wq, h Wk, h Wv; rotary
embedding of Q and K at the tokens' absolute positions (a replay from P
rotates exactly as the full run); attention through the paged pool (one pool
layer per model layer); x <- x + O Wo; h2 = RMSNorm(x) g_mlp;
x <- x + (SiLU(h2 Wg) * (h2 Wu)) Wd.  Every step is a library call; this
module only sequences them and owns scratch tensors.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import torch

from . import _native as N
from .pool import KVPool, gemm_bf16


def _stream(stream):
    return (stream or torch.cuda.current_stream()).cuda_stream


def rmsnorm(x: torch.Tensor, gain: torch.Tensor, eps: float, out: Optional[torch.Tensor] = None, stream=None):
    out = torch.empty_like(x) if out is None else out
    N.check(N.lib.pgsr_rmsnorm_bf16(x.shape[0], x.shape[1], x.data_ptr(), gain.data_ptr(), float(eps),
                                    out.data_ptr(), _stream(stream)))
    return out


def rope_(x: torch.Tensor, positions: torch.Tensor, theta: float, stream=None) -> torch.Tensor:
    """In place on x [n, heads, d]; positions: int32 [n] on the GPU."""
    assert positions.dtype == torch.int32 and positions.is_cuda
    N.check(N.lib.pgsr_rope_bf16(x.shape[0], x.shape[1], x.shape[2], x.data_ptr(), positions.data_ptr(),
                                 float(theta), _stream(stream)))
    return x


def silu_mul(gate_up: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    n, two_ff = gate_up.shape
    out = torch.empty((n, two_ff // 2), dtype=gate_up.dtype, device=gate_up.device) if out is None else out
    N.check(N.lib.pgsr_silu_mul_bf16(n, two_ff // 2, gate_up.data_ptr(), out.data_ptr(), _stream(stream)))
    return out


class DecoderReplay:
    def __init__(self, weights: Sequence[Dict[str, torch.Tensor]], n_q_heads: int, n_kv_heads: int,
                 head_dim: int, eps: float, theta: float, n_blocks: int, max_seqs: int,
                 max_blocks_per_seq: int, block_size: int = 16, workspace_bytes: int = 0):
        """``weights``: per layer a dict of bf16 CUDA tensors in the linear-layer
        [out][in] layout: wq [Hq*d, dm], wk, wv [Hkv*d, dm], wo [dm, Hq*d],
        w_gate_up [2*d_ff, dm] (gate rows then up rows), w_down [dm, d_ff],
        and the gains g_attn, g_mlp [dm]."""
        self.w = list(weights)
        self.hq, self.hkv, self.d, self.eps, self.theta = n_q_heads, n_kv_heads, head_dim, eps, theta
        self.d_model = self.w[0]["wq"].shape[1]
        self.d_ff = self.w[0]["w_down"].shape[1]
        self.pool = KVPool(len(self.w), n_q_heads, n_kv_heads, head_dim, n_blocks, max_seqs,
                           max_blocks_per_seq, N.BF16, block_size, workspace_bytes=workspace_bytes)
        self._buf: Dict[str, torch.Tensor] = {}

    def _scratch(self, name: str, *shape) -> torch.Tensor:
        n = 1
        for s in shape:
            n *= s
        t = self._buf.get(name)
        if t is None or t.numel() < n:
            t = self._buf[name] = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        return t[:n].view(*shape)

    def _run(self, fn, seq: int, x: torch.Tensor, pos0: int) -> torch.Tensor:
        n = x.shape[0]
        pos = torch.arange(pos0, pos0 + n, dtype=torch.int32, device="cuda")
        h = self._scratch("h", n, self.d_model)
        q = self._scratch("q", n, self.hq, self.d)
        k = self._scratch("k", n, self.hkv, self.d)
        v = self._scratch("v", n, self.hkv, self.d)
        o = self._scratch("o", n, self.hq * self.d)
        gu = self._scratch("gu", n, 2 * self.d_ff)
        a = self._scratch("a", n, self.d_ff)
        x = x.clone()
        scale = self.d ** -0.5
        last = len(self.w) - 1
        for li, w in enumerate(self.w):
            rmsnorm(x, w["g_attn"], self.eps, out=h)
            gemm_bf16(h, w["wq"], out=q.view(n, -1))
            gemm_bf16(h, w["wk"], out=k.view(n, -1))
            gemm_bf16(h, w["wv"], out=v.view(n, -1))
            rope_(q, pos, self.theta)
            rope_(k, pos, self.theta)
            rc = fn(li, [seq], [n], q, k, v, o, scale, commit=(li == last))
            if rc:
                raise N.PgsrError(rc, N.lib.pgsr_last_error().decode())
            gemm_bf16(o, w["wo"], r=x, out=x)                 # x <- x + O Wo
            rmsnorm(x, w["g_mlp"], self.eps, out=h)
            gemm_bf16(h, w["w_gate_up"], out=gu)
            silu_mul(gu, out=a)
            gemm_bf16(a, w["w_down"], r=x, out=x)             # x <- x + MLP(x)
        return x

    def replay(self, seq: int, x: torch.Tensor) -> torch.Tensor:
        """Tokens at positions len(seq) .. len(seq)+n-1 (Algorithm 1, replay loop)."""
        return self._run(self.pool.replay, seq, x, self.pool.seq_len(seq))

    def full_reset(self, seq: int, x: torch.Tensor) -> torch.Tensor:
        """Baseline B5: crop to 0 on the first layer, then all of x from position 0."""
        return self._run(self.pool.full_reset, seq, x, 0)

    def crop(self, seqs: List[int], new_lens: List[int]) -> int:
        return self.pool.crop(seqs, new_lens)

    def capture_restore_replay(self, seq: int, crop_len: int, x: torch.Tensor) -> "CapturedReplay":
        """Record the restore (crop of ``seq`` to ``crop_len``) and the replay
        of ``x`` through every layer as one HIP graph, from the pool state at
        this call.  Every library call of the two steps only enqueues kernels
        (no allocation, copy or memset on the stream), so the graph holds the
        launches the calls made, with the block ids the host mirror chose for
        that state.  Nothing runs during the capture: afterwards the host
        mirror reflects the recorded calls while the device is unchanged.
        Replaying is valid only from the captured state: restore it (device
        tables and host mirror, e.g. ``pool.load_meta``) before each replay."""
        n = x.shape[0]
        # scratch of its own, allocated before the capture and owned by the
        # result: the graph keeps these addresses, so eager calls that later
        # grow the shared scratch must not free them
        shared, self._buf = self._buf, {}
        try:
            for name, shape in (("h", (n, self.d_model)), ("q", (n, self.hq, self.d)),
                                ("k", (n, self.hkv, self.d)), ("v", (n, self.hkv, self.d)),
                                ("o", (n, self.hq * self.d)), ("gu", (n, 2 * self.d_ff)), ("a", (n, self.d_ff))):
                self._scratch(name, *shape)
            xin = x.clone()
            stream = torch.cuda.Stream()
            stream.wait_stream(torch.cuda.current_stream())
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.stream(stream):
                with torch.cuda.graph(graph, stream=stream):
                    rc = self.crop([seq], [crop_len])
                    if rc:
                        raise N.PgsrError(rc, N.lib.pgsr_last_error().decode())
                    out = self._run(self.pool.replay, seq, xin, crop_len)
            torch.cuda.current_stream().wait_stream(stream)
            own = self._buf
        finally:
            self._buf = shared
        return CapturedReplay(graph, xin, out, own)


class CapturedReplay:
    """A restore + replay recorded by DecoderReplay.capture_restore_replay:
    ``input`` holds the replayed token states (overwrite it in place to replay
    others), ``output`` receives the result of each ``replay()``."""

    def __init__(self, graph: "torch.cuda.CUDAGraph", inp: torch.Tensor, out: torch.Tensor,
                 scratch: Dict[str, torch.Tensor]):
        self.graph, self.input, self.output, self._scratch = graph, inp, out, scratch

    def replay(self) -> torch.Tensor:
        self.graph.replay()
        return self.output
