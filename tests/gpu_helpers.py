"""Helpers shared by the GPU parity tests: moving seeded episodes to the
device, driving the library through the C ABI, reading the paged pool back,
and the tolerance metrics (max |d| and L1-relative error sum|d| / sum|ref|)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads as W


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def dev(arr: np.ndarray, dtype: str) -> torch.Tensor:
    """Storage array from workloads (float32 or bf16 bits) -> CUDA tensor."""
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().contiguous().cpu()
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.view(torch.int32).numpy()


def storage_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    return (arr if dtype == "f32" else W.bf16_bits_to_f32(arr)).astype(np.float64)


def logical_kv(pool, layer: int, seq: int, n: int):
    """Logical K, V [n, Hkv, d] of tokens 0..n-1 of ``seq``, through the device table."""
    torch.cuda.synchronize()
    tables = pool.block_tables[seq].long()
    pos = torch.arange(n, device="cuda")
    blk, slot = tables[pos // pool.B], pos % pool.B
    k = pool.k_cache[layer][blk, :, slot, :]          # K: [block][head][slot][d]
    v = pool.v_cache[layer][blk, :, :, slot]          # V: [block][head][d][slot]
    return k, v


def errors(got: np.ndarray, ref: np.ndarray):
    d = np.abs(got.astype(np.float64) - ref)
    return float(d.max()) if d.size else 0.0, float(d.sum() / max(np.abs(ref).sum(), 1e-300))


def assert_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "") -> None:
    mx, rel = errors(got, ref)
    if dtype == "f32":
        assert mx <= 1e-4, f"{what}: max|d| {mx:.3e} > 1e-4"
    else:
        assert mx <= 2e-2 and rel <= 1e-2, f"{what}: max|d| {mx:.3e} (<= 2e-2), rel {rel:.3e} (<= 1e-2)"


def make_pool(geom: W.AttnGeometry, dtype: str, n_blocks: int, max_seqs: int, max_bps: int,
              n_layers: int = 1, block_size: int = 16, init_free_order=None, split_q: int = 0,
              max_splits: int = 16):
    """``split_q`` > 0 gives the pool a workspace for split-key replays of up
    to that many query tokens per call, in up to ``max_splits`` splits."""
    from paper_2609_04875_amd import KVPool, F32, BF16, workspace_bytes
    ws = workspace_bytes(geom.n_q_heads, geom.head_dim, split_q, max_splits) if split_q else 0
    return KVPool(n_layers, geom.n_q_heads, geom.n_kv_heads, geom.head_dim, n_blocks, max_seqs,
                  max_bps, F32 if dtype == "f32" else BF16, block_size, init_free_order,
                  workspace_bytes=ws)


def contaminated_then_crop(pool, ep: W.Episode, seq: int, scale: float, poison: bool = False):
    """Prefill the contaminated run of ``ep`` into ``seq``, then crop to its prefix.

    Returns the contaminated run's output (device)."""
    dt = ep.dtype
    cq, ck, cv = (dev(ep.contaminated(x), dt) for x in ("q", "k", "v"))
    co = torch.empty_like(cq)
    rc = pool.replay(0, [seq], [ep.t_contaminated], cq, ck, cv, co, scale)
    assert rc == 0, rc
    rc = pool.crop([seq], [ep.prefix], poison=poison)
    assert rc == 0, rc
    return co


def oracle_suffix(ep: W.Episode, scale: float, rows=None) -> np.ndarray:
    """fp64 oracle output of the sanitized suffix (queries at prefix .. T-1)."""
    q = storage_f64(ep.q[ep.prefix:], ep.dtype)
    k = storage_f64(ep.k, ep.dtype)
    v = storage_f64(ep.v, ep.dtype)
    return oracle.attention(q, k, v, ep.prefix, scale, rows=rows)
