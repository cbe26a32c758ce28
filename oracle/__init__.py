"""Plain CPU oracle of selective replay's hot path.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg import this package.  It shares no code with ``paper_2609_04875_amd`` and
never imports it; the two meet only in the seeded generators of ``workloads``.

Contents, each following the paper's definitions:

* :class:`PoolModel` -- the paged KV cache's block table and free-list stack.
  Restore of a checkpoint is a crop of the cache to the clean boundary
  (Section 3.4 (b), Algorithm 1 restore step; "cropping is restoring", Lemma 1);
  the replay loop of Algorithm 1 appends the sanitized suffix.  Paging itself is
  not in the paper; the readings below fix it.
* :func:`attention` -- fp64 prefix + causal softmax attention (C, see
  ``pgsr_oracle.c``): the prefill form of F (Eq. (1)) over the suffix.
* :func:`bf16_round` -- round-to-nearest-even to bfloat16, from the format's
  definition (8 significant bits).
* :func:`e4m3_round` -- rounding to FP8 E4M3 for the FP8 KV pool (F1, F2).
* :func:`stacked_layers` -- the stacked random-init layer F used by the 70B-like
  workload (a reading: the paper defines no layer).
* :func:`recomputed_transitions`, :func:`replay_gain` -- Corollary 1.

Readings where the paper is silent (it never describes paging):
  R1 block-table sentinel is -1 for logical blocks >= ceil(len / B);
  R2 the free list is a LIFO stack: push ``free[top++] = id``, pop
     ``id = free[--top]``; the default initial stack makes pops yield 0, 1, 2, ...;
  R3 a crop processes sequences in call order and, within one, pushes the freed
     ids in ascending logical-block order; a crop to the current length is a
     no-op, a crop to 0 frees every block; duplicates / out-of-range are errors
     and change nothing (all-or-nothing);
  R4 a reservation pops, per sequence in call order, the blocks for logical
     indices nalloc .. ceil((len + S) / B) - 1 in increasing order;
  R5 copy-on-write fork (all methods branch from one contaminated base,
     Section 4.1): a fork gives an empty sequence the source's table row and
     length, and every block counts the table entries that name it.  A crop
     releases an entry by decrementing its block's count and pushes the block
     only when the count reaches 0 (same order as R3).  A reservation that
     would write into a partial tail block (len mod B != 0, S > 0) named by more
     than one entry first pops a private block, copies the tail block's first
     len mod B slots of every layer into it, and puts it in the row (the old
     block's count drops by 1); this pop comes before the R4 pops.  The
     sequences of one reservation are taken in call order, each seeing the
     counts the earlier ones left (as in R3 and R4), so the last row still
     naming a shared tail writes into it without a copy.  Without forks every
     count is 0 or 1 and R3/R4 are unchanged.

Readings of the FP8 KV cache variant (the paper stores the cache at model
precision; the variant halves the bytes a decode step reads):
  F1 E4M3 rounding is round-to-nearest, ties to even, saturating: magnitudes
     past the largest finite value 448 store as +-448 (infinities too), NaN
     stays NaN (:func:`e4m3_round`);
  F2 each layer has one K scale and one V scale (positive, finite); a value x
     (bf16 from the projection) is stored as the code e4m3(fp32(x / scale)),
     with fp32 the correctly rounded quotient, and read back as code * scale;
     attention runs on the read-back values.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import build as _build

OK, EINVAL, ERANGE, ENOMEM = 0, 1, 2, 3

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        f = lib.pgsr_oracle_attention
        f.restype = ctypes.c_int
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        f.argtypes = [i64, i64, i64, i32, i32, i32, P, P, P, ctypes.c_double, P, i64, P]
        lib.pgsr_oracle_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the C oracle uses (OMP_NUM_THREADS, else all cores)."""
    return int(_load().pgsr_oracle_threads())


# --------------------------------------------------------------------------- #
# attention                                                                    #
# --------------------------------------------------------------------------- #
def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, pos0: int, scale: float,
              rows: Optional[np.ndarray] = None) -> np.ndarray:
    """fp64 prefix + causal attention.

    q [n_q, Hq, d] holds queries at absolute positions pos0 .. pos0 + n_q - 1;
    k, v [n_kv, Hkv, d] hold keys/values at positions 0 .. n_kv - 1 (the logical
    cache: cropped prefix followed by the replayed tokens).  Query head h reads
    KV head h // (Hq / Hkv).  ``rows`` (optional) lists flat indices i * Hq + h to
    evaluate; the result is then [len(rows), d] instead of [n_q, Hq, d].
    """
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    n_q, hq, d = q.shape
    n_kv, hkv, d2 = k.shape
    if d2 != d or v.shape != k.shape:
        raise ValueError("shape mismatch")
    if rows is None:
        out = np.empty((n_q, hq, d), np.float64)
        rows_p, n_rows = None, 0
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        out = np.empty((rows.shape[0], d), np.float64)
        rows_p, n_rows = rows.ctypes.data, rows.shape[0]
    rc = _load().pgsr_oracle_attention(n_q, pos0, n_kv, hq, hkv, d, q.ctypes.data, k.ctypes.data,
                                       v.ctypes.data, float(scale), rows_p, n_rows, out.ctypes.data)
    if rc != 0:
        raise ValueError(f"oracle attention rejected its arguments (status {rc})")
    return out


# --------------------------------------------------------------------------- #
# bf16 rounding from the format's definition                                   #
# --------------------------------------------------------------------------- #
def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits (1 implicit + 7 stored) and fp32's
    exponent range: normals down to 2**-126, subnormal spacing 2**-133,
    largest finite (2 - 2**-7) * 2**127.  Done directly from fp64 (one rounding).
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    fin = np.isfinite(x) & (x != 0)
    xf = x[fin]
    _, e = np.frexp(np.abs(xf))               # |x| = m * 2**e, m in [0.5, 1)
    lsb_exp = np.maximum(e - 8, -133)          # exponent of the last kept bit
    q = np.rint(np.ldexp(xf, -lsb_exp))        # rint: round half to even
    r = np.ldexp(q, lsb_exp)
    big = np.abs(r) > (2.0 - 2.0 ** -7) * 2.0 ** 127
    r[big] = np.copysign(np.inf, r[big])
    out[fin] = r
    out[~fin] = x[~fin]
    return out


# --------------------------------------------------------------------------- #
# block table + free list                                                      #
# --------------------------------------------------------------------------- #
E4M3_MAX = 448.0


def e4m3_round(x: np.ndarray) -> np.ndarray:
    """Round to the FP8 format E4M3 (OCP "e4m3fn": 1 sign, 4 exponent bits with
    bias 7, 3 mantissa bits, subnormal step 2^-9, largest finite 448, no
    infinities), to nearest with ties to even, from the format's definition.
    Reading F1 (FP8 KV cache): magnitudes past 448 saturate to 448 (infinities
    too); NaN stays NaN."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), 2 * E4M3_MAX)     # anything this large saturates; keeps inf out
    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.maximum(np.floor(np.log2(np.where(a > 0, a, 1.0))), -6.0)   # binade, subnormals at -6
        q = np.exp2(e - 3.0)                                                  # 3 mantissa bits
        r = np.rint(a / q) * q                                                # ties to even
    r = np.where(a > 0, r, 0.0)
    r = np.minimum(r, E4M3_MAX)
    return np.where(np.isnan(x), np.nan, np.copysign(r, x))


def _cdiv(a: int, b: int) -> int:
    return -(-a // b)


class PoolModel:
    """Host model of the paged KV pool's metadata (and, optionally, its data).

    tables [max_seqs, max_blocks]  int32, -1 = empty (R1)
    lens   [max_seqs]              committed tokens per sequence
    nalloc [max_seqs]              blocks held per row (>= ceil(len/B); larger
                                   while a reserved replay step is uncommitted)
    free   [n_blocks]              stack storage; free[0 .. top) are free ids (R2)
    refs   [n_blocks]              table entries naming each block (R5)
    """

    def __init__(self, n_blocks: int, max_seqs: int, max_blocks: int, block_size: int,
                 init_free_order: Optional[Sequence[int]] = None,
                 n_layers: int = 0, n_kv_heads: int = 0, head_dim: int = 0, kv_fp8: bool = False):
        self.B = block_size
        self.kv_fp8 = kv_fp8                 # store codes (F1, F2); scales per layer
        self.k_scales = np.ones(max(n_layers, 1))
        self.v_scales = np.ones(max(n_layers, 1))
        self.n_blocks = n_blocks
        self.tables = np.full((max_seqs, max_blocks), -1, np.int32)
        self.lens = np.zeros(max_seqs, np.int32)
        self.nalloc = np.zeros(max_seqs, np.int32)
        if init_free_order is None:
            self.free = np.arange(n_blocks - 1, -1, -1, dtype=np.int32)
        else:
            self.free = np.array(init_free_order, dtype=np.int32)
            if sorted(self.free.tolist()) != list(range(n_blocks)):
                raise ValueError("init_free_order must be a permutation of the block ids")
        self.top = n_blocks
        self.refs = np.zeros(n_blocks, np.int32)
        # optional data: [layer][block][slot][kv_head][d], fp64 (oracle's own layout)
        self.kdata = self.vdata = None
        if n_layers:
            shape = (n_layers, n_blocks, block_size, n_kv_heads, head_dim)
            self.kdata = np.full(shape, np.nan)
            self.vdata = np.full(shape, np.nan)

    # -- validation shared by the calls (all-or-nothing) --
    def _check_seqs(self, seqs: Sequence[int]) -> int:
        if len(set(seqs)) != len(seqs):
            return EINVAL
        for s in seqs:
            if not (0 <= s < self.tables.shape[0]):
                return EINVAL
        return OK

    def crop(self, seqs: Sequence[int], new_lens: Sequence[int]) -> int:
        """Restore = crop (Algorithm 1 restore step): keep new_lens[i] tokens."""
        if len(seqs) != len(new_lens):
            return EINVAL
        rc = self._check_seqs(seqs)
        if rc:
            return rc
        for s, L in zip(seqs, new_lens):
            if L < 0 or L > self.lens[s]:
                return ERANGE
        for s, L in zip(seqs, new_lens):
            keep = _cdiv(L, self.B)
            for j in range(keep, int(self.nalloc[s])):       # ascending logical order (R3)
                b = int(self.tables[s, j])
                self.tables[s, j] = -1
                self.refs[b] -= 1
                if self.refs[b] == 0:                         # last entry naming it (R5)
                    self.free[self.top] = b
                    self.top += 1
            self.nalloc[s] = keep
            self.lens[s] = L
        return OK

    def _shared_tail(self, s: int, S: int) -> bool:
        """R5: the next write lands in a partial tail block other entries name."""
        L = int(self.lens[s])
        return S > 0 and L % self.B != 0 and int(self.refs[self.tables[s, L // self.B]]) > 1

    def fork(self, srcs: Sequence[int], dsts: Sequence[int]) -> int:
        """Copy-on-write fork (R5): each empty dsts[i] shares srcs[i]'s blocks."""
        if len(srcs) != len(dsts):
            return EINVAL
        for ids in (srcs, dsts):
            for x in ids:
                if not (0 <= x < self.tables.shape[0]):
                    return EINVAL
        if len(set(dsts)) != len(dsts) or set(dsts) & set(srcs):
            return EINVAL
        for d in dsts:
            if self.lens[d] != 0 or self.nalloc[d] != 0:
                return EINVAL
        for s, d in zip(srcs, dsts):
            n = int(self.nalloc[s])
            self.tables[d, :n] = self.tables[s, :n]
            self.nalloc[d] = n
            self.lens[d] = self.lens[s]
            for b in self.tables[s, :n]:
                self.refs[b] += 1
        return OK

    def reserve(self, seqs: Sequence[int], q_lens: Sequence[int]) -> int:
        """Pop the blocks that positions len .. len+S-1 need (R4)."""
        if len(seqs) != len(q_lens):
            return EINVAL
        rc = self._check_seqs(seqs)
        if rc:
            return rc
        need = []
        for s, S in zip(seqs, q_lens):
            if S < 0:
                return EINVAL
            blocks = _cdiv(int(self.lens[s]) + S, self.B)
            if blocks > self.tables.shape[1]:
                return ERANGE
            need.append(max(0, blocks - int(self.nalloc[s])))
        # copies needed, in call order: each one releases an entry of its tail block (R5)
        refs_left = {}
        n_cow = 0
        for s, S in zip(seqs, q_lens):
            L = int(self.lens[s])
            if S > 0 and L % self.B != 0:
                b = int(self.tables[s, L // self.B])
                r = refs_left.get(b, int(self.refs[b]))
                if r > 1:
                    n_cow += 1
                    refs_left[b] = r - 1
        if sum(need) + n_cow > self.top:
            return ENOMEM
        for s, S, n in zip(seqs, q_lens, need):
            if self._shared_tail(s, S):                       # private copy of the tail block (R5)
                j = int(self.lens[s]) // self.B
                old = int(self.tables[s, j])
                self.top -= 1
                new = int(self.free[self.top])
                if self.kdata is not None:
                    t = int(self.lens[s]) % self.B
                    self.kdata[:, new, :t] = self.kdata[:, old, :t]
                    self.vdata[:, new, :t] = self.vdata[:, old, :t]
                self.tables[s, j] = new
                self.refs[old] -= 1
                self.refs[new] = 1
            for _ in range(n):
                self.top -= 1
                b = int(self.free[self.top])
                self.tables[s, self.nalloc[s]] = b
                self.refs[b] = 1
                self.nalloc[s] += 1
        return OK

    def commit(self, seqs: Sequence[int], q_lens: Sequence[int]) -> None:
        for s, S in zip(seqs, q_lens):
            self.lens[s] += S

    def slot(self, seq: int, pos: int) -> Tuple[int, int]:
        """Physical (block id, offset) of logical token ``pos`` of ``seq``."""
        return int(self.tables[seq, pos // self.B]), pos % self.B

    # -- data (oracle's own layout) --
    def set_kv_scales(self, k_scales: Sequence[float], v_scales: Sequence[float]) -> None:
        """F2: one K and one V scale per layer (fp32 values)."""
        self.k_scales = np.asarray(k_scales, dtype=np.float32).astype(np.float64)
        self.v_scales = np.asarray(v_scales, dtype=np.float32).astype(np.float64)

    def quantize(self, x: np.ndarray, scale: float) -> np.ndarray:
        """F2: the code values (as fp64) stored for x, e4m3(fp32(x / scale))."""
        q = np.asarray(x, dtype=np.float64).astype(np.float32) / np.float32(scale)   # fp32 quotient
        return e4m3_round(q.astype(np.float64))

    def write(self, layer: int, seq: int, start: int, k: np.ndarray, v: np.ndarray) -> None:
        if self.kv_fp8:
            k = self.quantize(k, self.k_scales[layer])
            v = self.quantize(v, self.v_scales[layer])
        for t in range(k.shape[0]):
            b, o = self.slot(seq, start + t)
            self.kdata[layer, b, o] = k[t]
            self.vdata[layer, b, o] = v[t]

    def gather(self, layer: int, seq: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
        """Logical K, V of tokens 0 .. n-1 of ``seq`` read through the block table
        (FP8 pools: code * scale, F2)."""
        idx = [self.slot(seq, p) for p in range(n)]
        k = np.stack([self.kdata[layer, b, o] for b, o in idx]) if n else np.zeros((0,) + self.kdata.shape[3:])
        v = np.stack([self.vdata[layer, b, o] for b, o in idx]) if n else np.zeros((0,) + self.vdata.shape[3:])
        if self.kv_fp8:
            k, v = k * self.k_scales[layer], v * self.v_scales[layer]
        return k, v

    def state(self) -> Dict[str, np.ndarray]:
        return {"tables": self.tables.copy(), "lens": self.lens.copy(),
                "free": self.free.copy(), "top": np.int32(self.top), "refs": self.refs.copy()}


def prefill(pool: PoolModel, layer: int, seqs: Sequence[int], q_lens: Sequence[int],
            q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
            commit: bool = True) -> List[np.ndarray]:
    """One replay call on the oracle pool: reserve, write K/V, attend, commit.

    q/k/v are packed in ``seqs`` order ([sum S, H, d]).  Returns the per-sequence
    outputs [S_i, Hq, d] (fp64).
    """
    rc = pool.reserve(seqs, q_lens)
    if rc:
        raise ValueError(f"reserve failed with status {rc}")
    outs, off = [], 0
    for s, S in zip(seqs, q_lens):
        P = int(pool.lens[s])
        pool.write(layer, s, P, k[off:off + S], v[off:off + S])
        kk, vv = pool.gather(layer, s, P + S)
        outs.append(attention(q[off:off + S], kk, vv, P, scale))
        off += S
    if commit:
        pool.commit(seqs, q_lens)
    return outs


# --------------------------------------------------------------------------- #
# Corollary 1                                                                  #
# --------------------------------------------------------------------------- #
def recomputed_transitions(T: int, tau: int) -> int:
    """Transitions F runs in a replay from boundary tau - 1: T - tau + 1 (Corollary 1)."""
    if not (1 <= tau <= T + 1):
        raise ValueError("tau must satisfy 1 <= tau <= T + 1")
    return T - tau + 1


def replay_gain(T: int, tau: int) -> float:
    """Gain over a full reset (T transitions): T / (T - tau + 1) (Corollary 1)."""
    return T / recomputed_transitions(T, tau)


# --------------------------------------------------------------------------- #
# stacked random-init layers (reading: the paper defines no layer)            #
# --------------------------------------------------------------------------- #
def stacked_layers(x: np.ndarray, layers, n_q_heads: int, n_kv_heads: int, head_dim: int,
                   scale: float, pos0: int = 0, cache: Optional[List[Tuple[np.ndarray, np.ndarray]]] = None,
                   record: Optional[list] = None):
    """F for the stacked workload: per layer, with bf16 storage points mirrored,

        Q = bf16(x Wq), K = bf16(x Wk), V = bf16(x Wv)
        O = bf16(attention(Q, [K_cache; K], [V_cache; V]))     (queries at pos0 ..)
        x = bf16(x + O Wo)

    ``x`` [n, d_model] are the token states at positions pos0 .. pos0+n-1 (fp64
    holding bf16 values); ``layers`` is a list of (Wq, Wk, Wv, Wo) fp64 arrays;
    ``cache`` gives each layer's K/V for positions 0 .. pos0-1 (the cropped
    prefix), or None when pos0 == 0.  Returns (x_out, per-layer (K, V) of the
    n new tokens).  Matrix products are library matmuls in fp64.  ``record``
    (a list), when given, receives each layer's O [n, Hq * d].
    """
    n = x.shape[0]
    new_kv = []
    for li, (wq, wk, wv, wo) in enumerate(layers):
        q = bf16_round(x @ wq).reshape(n, n_q_heads, head_dim)
        k = bf16_round(x @ wk).reshape(n, n_kv_heads, head_dim)
        v = bf16_round(x @ wv).reshape(n, n_kv_heads, head_dim)
        if pos0 > 0:
            kc, vc = cache[li]
            kk, vv = np.concatenate([kc[:pos0], k]), np.concatenate([vc[:pos0], v])
        else:
            kk, vv = k, v
        o = bf16_round(attention(q, kk, vv, pos0, scale)).reshape(n, n_q_heads * head_dim)
        if record is not None:
            record.append(o)
        x = bf16_round(x + o @ wo)
        new_kv.append((k, v))
    return x, new_kv
