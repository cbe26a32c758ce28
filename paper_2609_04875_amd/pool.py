"""Paged KV pool over torch device memory, driving the C ABI.

``KVPool`` allocates the caller-owned device arrays the library works on
(caches, block table, lengths, free-list stack, split workspace) and exposes
the three calls of the hot path: ``crop`` (restore, Algorithm 1), ``replay``
(the prefill form of the replay loop) and ``full_reset`` (baseline B5).
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import torch

from . import _native as N

# (cache storage dtype, dtype of q / k / v / o) per pool dtype; an FP8 pool
# holds raw E4M3 codes as bytes.
_DT = {N.F32: (torch.float32, torch.float32), N.BF16: (torch.bfloat16, torch.bfloat16),
       N.FP8_E4M3: (torch.uint8, torch.bfloat16)}


def _stream_ptr(stream: Optional[torch.cuda.Stream], device: Optional[int] = None) -> Optional[int]:
    """Raw HIP stream handle: the given stream, else torch's current stream on
    ``device`` (read without building a Stream object, which costs several
    microseconds per call)."""
    if stream is not None:
        return stream.cuda_stream or None
    idx = torch.cuda.current_device() if device is None else device
    return torch._C._cuda_getCurrentRawStream(idx) or None


def _dev_ptr(t: Optional[torch.Tensor], dtype, name: str, device: Optional[int] = None,
             numel: Optional[int] = None) -> Optional[int]:
    """Device address of ``t`` after checking what the C ABI cannot: dtype,
    contiguity, that it is on ``device`` (when given) and holds exactly
    ``numel`` elements (when given).  The library takes raw pointers, so a
    short tensor would otherwise be read or written past its end."""
    if t is None:
        if numel:
            raise ValueError(f"{name} is None but {numel} elements are needed")
        return None
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} holds {t.numel()} elements; the call needs exactly {numel}")
    if not t.is_cuda or not t.is_contiguous() or t.dtype != dtype:
        raise ValueError(f"{name} must be a contiguous {dtype} CUDA tensor")
    if device is not None and t.device.index != device:
        raise ValueError(f"{name} is on cuda:{t.device.index}; the pool is on cuda:{device}")
    return t.data_ptr() if t.numel() else None


def prefill_sizes(n_q_heads: int, n_kv_heads: int, head_dim: int, q_lens: Sequence[int]):
    """Elements that q / o and k / v of a prefill call must hold:
    sum(q_lens) tokens of [n_q_heads][head_dim] and [n_kv_heads][head_dim]."""
    tot = sum(int(x) for x in q_lens)
    return tot * n_q_heads * head_dim, tot * n_kv_heads * head_dim


class KVPool:
    def __init__(self, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 n_blocks: int, max_seqs: int, max_blocks_per_seq: int, dtype: int = N.BF16,
                 block_size: int = 16, init_free_order: Optional[Sequence[int]] = None,
                 workspace_bytes: int = 0, device: str = "cuda",
                 stream: Optional[torch.cuda.Stream] = None):
        self.n_layers, self.hq, self.hkv, self.d = n_layers, n_q_heads, n_kv_heads, head_dim
        self.n_blocks, self.max_seqs, self.max_bps = n_blocks, max_seqs, max_blocks_per_seq
        self.B, self.dtype_code = block_size, dtype
        self.cache_dtype, self.dtype = _DT[dtype]
        shape = (n_layers, n_blocks, n_kv_heads, block_size, head_dim)
        self.k_cache = torch.zeros(shape, dtype=self.cache_dtype, device=device)
        self.v_cache = torch.zeros((n_layers, n_blocks, n_kv_heads, head_dim, block_size),
                                   dtype=self.cache_dtype, device=device)
        self.block_tables = torch.empty((max_seqs, max_blocks_per_seq), dtype=torch.int32, device=device)
        self.seq_lens = torch.empty((max_seqs,), dtype=torch.int32, device=device)
        self.free_list = torch.empty((n_blocks,), dtype=torch.int32, device=device)
        self.free_top = torch.empty((1,), dtype=torch.int32, device=device)
        self.ref_counts = torch.empty((n_blocks,), dtype=torch.int32, device=device)
        self.workspace = (torch.empty((workspace_bytes,), dtype=torch.uint8, device=device)
                          if workspace_bytes else None)
        order = N.int32_array(init_free_order) if init_free_order is not None else None
        handle = ctypes.c_void_p()
        N.check(N.lib.pgsr_pool_create(
            n_layers, n_q_heads, n_kv_heads, head_dim, block_size, dtype, n_blocks, max_seqs,
            max_blocks_per_seq, self.k_cache.data_ptr(), self.v_cache.data_ptr(),
            self.block_tables.data_ptr(), self.seq_lens.data_ptr(), self.free_list.data_ptr(),
            self.free_top.data_ptr(), self.ref_counts.data_ptr(),
            self.workspace.data_ptr() if self.workspace is not None else None,
            workspace_bytes, order, _stream_ptr(stream), ctypes.byref(handle)))
        self._h = handle
        self._dev = self.k_cache.device.index
        self.recomputed_tokens = ctypes.c_int64(0)

    def close(self) -> None:
        if self._h:
            N.lib.pgsr_pool_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- host-mirror queries ----
    def seq_len(self, seq: int) -> int:
        out = ctypes.c_int32()
        N.check(N.lib.pgsr_seq_len(self._h, seq, ctypes.byref(out)))
        return out.value

    def free_blocks(self) -> int:
        out = ctypes.c_int32()
        N.check(N.lib.pgsr_free_blocks(self._h, ctypes.byref(out)))
        return out.value

    def refresh(self, stream=None) -> None:
        N.check(N.lib.pgsr_pool_refresh(self._h, _stream_ptr(stream, self._dev)))

    def set_kv_scales(self, k_scales: Sequence[float], v_scales: Sequence[float]) -> None:
        """Per-layer K and V scales of an FP8 pool (stored code = x / scale)."""
        if len(k_scales) != self.n_layers or len(v_scales) != self.n_layers:
            raise ValueError("one K and one V scale per layer")
        ks = (ctypes.c_float * self.n_layers)(*map(float, k_scales))
        vs = (ctypes.c_float * self.n_layers)(*map(float, v_scales))
        N.check(N.lib.pgsr_pool_set_kv_scales(self._h, ks, vs))

    def set_prefill_kernel(self, kind: str) -> None:
        """bf16 prefill kernel: "auto" (wide, else pipelined, where they apply),
        "pipelined" (never the wide kernel) or "four_wave"."""
        code = {"auto": 0, "four_wave": 1, "pipelined": 2}[kind]
        N.check(N.lib.pgsr_pool_set_prefill_kernel(self._h, code))

    # ---- kernel timing (HIP events recorded by the library on the call's stream) ----
    def enable_timing(self, on: bool = True) -> None:
        N.check(N.lib.pgsr_pool_enable_timing(self._h, 1 if on else 0))

    def last_times(self):
        """(append_ms, attention_ms) of the most recent replay / full-reset call."""
        a, b = ctypes.c_float(), ctypes.c_float()
        N.check(N.lib.pgsr_pool_last_times(self._h, ctypes.byref(a), ctypes.byref(b)))
        return a.value, b.value

    def set_clock_probe(self, workgroups: int = 0) -> None:
        """Shader-clock probe on the bf16 prefill launches of timed calls: a
        device buffer for ``workgroups`` workgroups (0 turns it off)."""
        self._clk = (torch.zeros((max(workgroups, 0) * 4,), dtype=torch.int64, device=self.k_cache.device)
                     if workgroups > 0 else None)
        N.check(N.lib.pgsr_pool_set_clock_buffer(
            self._h, self._clk.data_ptr() if self._clk is not None else None,
            self._clk.numel() * 8 if self._clk is not None else 0))

    def last_clock(self, stream=None):
        """(GHz, shader cycles, reference ticks) summed over the workgroups of
        the most recent timed prefill launch."""
        ghz, cyc, tck = ctypes.c_double(), ctypes.c_int64(), ctypes.c_int64()
        N.check(N.lib.pgsr_pool_last_clock(self._h, _stream_ptr(stream, self._dev), ctypes.byref(ghz),
                                           ctypes.byref(cyc), ctypes.byref(tck)))
        return ghz.value, cyc.value, tck.value

    # ---- the hot path ----
    def crop(self, seqs: Sequence[int], new_lens: Sequence[int], poison: bool = False,
             stream=None) -> int:
        """Restore = crop; returns the status (0 ok) instead of raising."""
        return N.lib.pgsr_kv_crop(self._h, len(seqs), N.int32_array(seqs), N.int32_array(new_lens),
                                  N.POISON if poison else 0, _stream_ptr(stream, self._dev))

    def fork(self, srcs: Sequence[int], dsts: Sequence[int], stream=None) -> int:
        """Copy-on-write fork of srcs[i] into the empty dsts[i]; returns the status."""
        return N.lib.pgsr_kv_fork(self._h, len(srcs), N.int32_array(srcs), N.int32_array(dsts),
                                  _stream_ptr(stream, self._dev))

    def _prefill(self, fn, layer, seqs, q_lens, q, k, v, o, scale, commit, stream) -> int:
        dt, dv = self.dtype, self._dev
        if len(q_lens) != len(seqs):
            raise ValueError(f"{len(seqs)} sequences but {len(q_lens)} lengths")
        if any(int(x) < 0 for x in q_lens):
            raise ValueError("negative query length")
        nq, nkv = prefill_sizes(self.hq, self.hkv, self.d, q_lens)
        return fn(self._h, layer, len(seqs), N.int32_array(seqs), N.int32_array(q_lens),
                  _dev_ptr(q, dt, "q", dv, nq), _dev_ptr(k, dt, "k", dv, nkv),
                  _dev_ptr(v, dt, "v", dv, nkv), _dev_ptr(o, dt, "o", dv, nq), float(scale),
                  N.COMMIT if commit else 0, ctypes.byref(self.recomputed_tokens),
                  _stream_ptr(stream, dv))

    def replay(self, layer: int, seqs, q_lens, q, k, v, o, scale: float, commit: bool = True,
               stream=None) -> int:
        return self._prefill(N.lib.pgsr_replay_prefill, layer, seqs, q_lens, q, k, v, o, scale,
                             commit, stream)

    def restore_replay(self, layer: int, seqs, restore_lens, q_lens, q, k, v, o, scale: float,
                       commit: bool = True, stream=None) -> int:
        """Restore (crop to ``restore_lens``) then replay ``q_lens`` tokens on
        ``layer``, in one call: the same result as ``crop`` then ``replay``,
        all-or-nothing across both; returns the status."""
        if len(restore_lens) != len(seqs):
            raise ValueError(f"{len(seqs)} sequences but {len(restore_lens)} restore lengths")
        rl = N.int32_array(restore_lens)
        return self._prefill(
            lambda h, layer_, n, s, ql, q_, k_, v_, o_, sc, fl, rec, st: N.lib.pgsr_restore_replay_prefill(
                h, layer_, n, s, rl, ql, q_, k_, v_, o_, sc, fl, rec, st),
            layer, seqs, q_lens, q, k, v, o, scale, commit, stream)

    def replay_static(self, layer: int, seqs, q_lens, q, k, v, o, scale: float, scratch_bytes: int,
                      commit: bool = True, stream=None) -> int:
        """``replay`` with the split / decode partials in the library's static
        device scratch instead of the pool's workspace (no allocation), as if
        the workspace were ``scratch_bytes`` large; returns the status."""
        return self._prefill(
            lambda h, layer_, n, s, ql, q_, k_, v_, o_, sc, fl, rec, st: N.lib.pgsr_replay_prefill_static(
                h, layer_, n, s, ql, q_, k_, v_, o_, sc, fl, int(scratch_bytes), rec, st),
            layer, seqs, q_lens, q, k, v, o, scale, commit, stream)

    def full_reset(self, layer: int, seqs, lens, q, k, v, o, scale: float, commit: bool = True,
                   stream=None) -> int:
        return self._prefill(N.lib.pgsr_full_reset_prefill, layer, seqs, lens, q, k, v, o, scale,
                             commit, stream)

    # ---- state snapshots (device -> host), for tests and the benchmark ----
    def state(self):
        torch.cuda.synchronize()
        return {"tables": self.block_tables.cpu().numpy(), "lens": self.seq_lens.cpu().numpy(),
                "free": self.free_list.cpu().numpy(), "top": int(self.free_top.item()),
                "refs": self.ref_counts.cpu().numpy()}

    def _meta(self):
        return (self.block_tables, self.seq_lens, self.free_list, self.free_top, self.ref_counts)

    def save_meta(self):
        return [t.clone() for t in self._meta()]

    def load_meta(self, saved) -> None:
        for dst, src in zip(self._meta(), saved):
            dst.copy_(src)
        self.refresh()


def workspace_bytes(n_q_heads: int, head_dim: int, max_total_q: int, max_splits: int = 16) -> int:
    """Workspace that lets replays of up to max_total_q query tokens split keys."""
    return int(N.lib.pgsr_workspace_bytes(n_q_heads, head_dim, max_total_q, max_splits))


def gemm_bf16(x: torch.Tensor, w: torch.Tensor, r: Optional[torch.Tensor] = None,
              out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Y = X W^T (+ R) on the library's MFMA GEMM, W in the [n][k] layout;
    bf16 in and out, fp32 accumulation."""
    m, k = x.shape
    n, k2 = w.shape
    if k2 != k:
        raise ValueError("inner dimensions differ")
    dv = x.device.index
    if out is None:
        out = torch.empty((m, n), dtype=torch.bfloat16, device=x.device)
    bf = torch.bfloat16
    N.check(N.lib.pgsr_gemm_bf16(m, n, k, _dev_ptr(x, bf, "x"), _dev_ptr(w, bf, "w", dv),
                                 _dev_ptr(r, bf, "r", dv, m * n) if r is not None else None,
                                 _dev_ptr(out, bf, "out", dv, m * n), _stream_ptr(stream, dv)))
    return out
