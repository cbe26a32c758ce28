"""Seeded synthetic episodes for selective replay.

This module only *draws* inputs. It holds none of the method's arithmetic: no
attention, no block-table logic, no crop. Both the fp64 oracle (``oracle/``)
and the HIP path (``paper_2609_04875_amd``) consume what it returns, and it
imports neither of them.

Model of an episode (the paper's transition system, Section 3.1, Eq. (1)):
one token is one transition. A contaminated run of ``t_contaminated`` tokens
was prefilled into the paged KV cache; the forget target entered at the
1-indexed step ``tau`` (Section 3.1), so positions ``0 .. tau-2`` are the clean
prefix (Lemma 1) and the crop keeps ``prefix = tau - 1`` tokens. The sanitized
suffix (Algorithm 1, the replay loop) has ``suffix`` tokens at absolute
positions ``prefix .. prefix + suffix - 1``; the counterfactual trajectory has
``t_sanitized = prefix + suffix`` tokens (Theorem 1).

Draw order for one episode, all fp32 N(0, 1) from ``numpy.random.default_rng``:
sanitized Q [T, Hq, d], sanitized K [T, Hkv, d], sanitized V [T, Hkv, d]
(positions 0 .. T-1), then the contaminated suffix Q, K, V
(positions prefix .. t_contaminated-1). Everything is then rounded once to the
workload dtype (round-to-nearest-even for bf16), so both sides see the same
bits. Contaminated positions below ``prefix`` are the sanitized ones: the two
runs share their prefix by construction.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

__all__ = [
    "Episode", "AttnGeometry", "Workload", "WORKLOADS", "workload",
    "draw_episode", "draw_ragged_lengths", "f32_to_bf16_bits", "bf16_bits_to_f32",
    "round_to_dtype", "stack_inputs",
]


# --------------------------------------------------------------------------- #
# dtype plumbing (storage only: fp32 -> bf16 round-to-nearest-even of inputs)  #
# --------------------------------------------------------------------------- #
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even) and return uint16 bits.

    Inputs drawn here are finite; NaN/inf are not produced by the generators.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    flat = u.reshape(-1)
    out = np.empty(flat.shape, np.uint16)
    step = 1 << 20                      # in cache-sized pieces, one scratch buffer
    tmp = np.empty(min(step, flat.size), np.uint32)
    for i in range(0, flat.size, step):
        src = flat[i:i + step]
        t = tmp[:src.size]
        np.right_shift(src, np.uint32(16), out=t)
        np.bitwise_and(t, np.uint32(1), out=t)          # lsb of the kept half: ties to even
        np.add(t, np.uint32(0x7FFF), out=t)
        np.add(t, src, out=t)
        np.right_shift(t, np.uint32(16), out=t)
        out[i:i + src.size] = t
    return out.reshape(u.shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bits (uint16) to the fp32 values they encode (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Storage array for ``dtype``: fp32 values as float32, bf16 as uint16 bits."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def _as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    return x if dtype == "f32" else bf16_bits_to_f32(x)


# --------------------------------------------------------------------------- #
# workload descriptions                                                        #
# --------------------------------------------------------------------------- #
@dataclasses.dataclass(frozen=True)
class AttnGeometry:
    n_q_heads: int
    n_kv_heads: int
    head_dim: int

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    """One named synthetic workload.

    ``prefix``/``suffix``/``t_contaminated`` describe a single episode; the ragged
    workload draws its episodes with :func:`draw_ragged_lengths` instead.
    """
    name: str
    geometry: AttnGeometry
    dtype: str                 # "f32" or "bf16": storage dtype of Q/K/V/O and the cache
    seed: int
    block_size: int = 16
    prefix: int = 0            # P = tau - 1, tokens kept by the crop
    suffix: int = 0            # S = T - tau + 1, replayed tokens
    t_contaminated: int = 0    # tokens in the contaminated cache before the crop
    n_episodes: int = 1
    chunk: int = 0             # > 0: replay the suffix in chunks of this many tokens
    n_layers: int = 1
    d_model: int = 0           # > 0: stacked random-init layers with projections
    prefix_fracs: Sequence[float] = ()   # stacked workload: crop points as fractions of T
    t_total: int = 0           # stacked workload: sanitized trajectory length
    softmax_scale: Optional[float] = None

    @property
    def t_sanitized(self) -> int:
        return self.prefix + self.suffix

    @property
    def scale(self) -> float:
        if self.softmax_scale is not None:
            return self.softmax_scale
        return 1.0 / float(np.sqrt(self.geometry.head_dim))


LLAMA8B = AttnGeometry(32, 8, 128)
SEVENTY_B = AttnGeometry(64, 8, 128)

WORKLOADS = {
    # Tiny single episode in fp32: MHA, 8 heads, d=64; 640 contaminated tokens,
    # target injected at 0-indexed position 512 (tau = 513): P = 512, S = 128.
    "tiny_mha8_d64_p512_s128_f32": Workload(
        "tiny_mha8_d64_p512_s128_f32", AttnGeometry(8, 8, 64), "f32", seed=0,
        prefix=512, suffix=128, t_contaminated=640),
    # Llama-3-8B attention geometry in bf16 (32q/8kv, d=128). The contaminated
    # cache holds 8192 + 2048 = 10240 tokens; the crop keeps 8189 tokens (not a
    # multiple of the 16-token block) and the 2048-token sanitized suffix is
    # replayed at positions 8189 .. 10236 (full reset: 10237 tokens).
    "llama8b_p8189_s2048_bf16": Workload(
        "llama8b_p8189_s2048_bf16", LLAMA8B, "bf16", seed=1,
        prefix=8189, suffix=2048, t_contaminated=10240),
    # 16 ragged episodes, T ~ U[4096, 16384], tau at U[10%, 90%] of T; one
    # shared pool, one varlen replay launch.
    "ragged16_llama8b_bf16": Workload(
        "ragged16_llama8b_bf16", LLAMA8B, "bf16", seed=2, n_episodes=16),
    # Long-horizon agent: 32768-token prefix, 4096-token suffix replayed in
    # 512-token chunks that each append to the cache before the next.
    "long32k_chunk512_llama8b_bf16": Workload(
        "long32k_chunk512_llama8b_bf16", LLAMA8B, "bf16", seed=3,
        prefix=32768, suffix=4096, t_contaminated=36864, chunk=512),
    # 70B-like geometry (64q/8kv, d=128), 8 stacked random-init attention
    # layers with d_model 8192; T = 16384, crop at 25/50/75/95 % of T.
    "stack70b_8layer_t16384_bf16": Workload(
        "stack70b_8layer_t16384_bf16", SEVENTY_B, "bf16", seed=4,
        n_layers=8, d_model=8192, t_total=16384,
        prefix_fracs=(0.25, 0.50, 0.75, 0.95)),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


# --------------------------------------------------------------------------- #
# episodes                                                                     #
# --------------------------------------------------------------------------- #
@dataclasses.dataclass
class Episode:
    """Inputs of one episode, already rounded to the storage dtype.

    ``q, k, v``      : sanitized trajectory, [T, H, d] (T = prefix + suffix)
    ``cq, ck, cv``   : contaminated suffix at positions prefix .. t_contaminated-1
    f32 storage is float32; bf16 storage is uint16 bits.
    """
    dtype: str
    prefix: int
    suffix: int
    t_contaminated: int
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    cq: np.ndarray
    ck: np.ndarray
    cv: np.ndarray

    @property
    def t_sanitized(self) -> int:
        return self.prefix + self.suffix

    # whole contaminated trajectory = shared prefix + contaminated suffix
    def contaminated(self, which: str) -> np.ndarray:
        base = {"q": self.q, "k": self.k, "v": self.v}[which]
        tail = {"q": self.cq, "k": self.ck, "v": self.cv}[which]
        return np.concatenate([base[: self.prefix], tail], axis=0)

    def as_f32(self, arr: np.ndarray) -> np.ndarray:
        return _as_f32(arr, self.dtype)


def _normal(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def draw_episode(rng: np.random.Generator, geom: AttnGeometry, dtype: str,
                 prefix: int, suffix: int, t_contaminated: int,
                 with_queries: bool = True) -> Episode:
    """Draw one episode in the documented order (see the module docstring).

    ``with_queries=False`` skips the query draws of the contaminated suffix
    (never needed to build a contaminated cache); the sanitized queries are
    always drawn so the draw order does not depend on the caller.
    """
    T = prefix + suffix
    if not (0 <= prefix <= t_contaminated):
        raise ValueError("prefix must lie inside the contaminated run")
    hq, hkv, d = geom.n_q_heads, geom.n_kv_heads, geom.head_dim
    q = _normal(rng, (T, hq, d))
    k = _normal(rng, (T, hkv, d))
    v = _normal(rng, (T, hkv, d))
    n_c = t_contaminated - prefix
    cq = _normal(rng, (n_c, hq, d)) if with_queries else np.zeros((n_c, hq, d), np.float32)
    ck = _normal(rng, (n_c, hkv, d))
    cv = _normal(rng, (n_c, hkv, d))
    r = lambda a: round_to_dtype(a, dtype)
    return Episode(dtype, prefix, suffix, t_contaminated, r(q), r(k), r(v), r(cq), r(ck), r(cv))


def single_episode(w: Workload) -> Episode:
    rng = np.random.default_rng(w.seed)
    return draw_episode(rng, w.geometry, w.dtype, w.prefix, w.suffix, w.t_contaminated)


def draw_ragged_lengths(seed: int, n: int, t_lo: int = 4096, t_hi: int = 16384,
                        f_lo: float = 0.10, f_hi: float = 0.90):
    """(T_i, P_i, S_i) for ``n`` ragged episodes, drawn first from the seed's stream.

    T_i ~ U{t_lo..t_hi} (inclusive); the injection fraction f_i ~ U[f_lo, f_hi);
    P_i = floor(f_i * T_i) tokens are kept, S_i = T_i - P_i are replayed
    (tau_i = P_i + 1). Returns the generator positioned after these draws.
    """
    rng = np.random.default_rng(seed)
    lens = []
    for _ in range(n):
        t = int(rng.integers(t_lo, t_hi, endpoint=True))
        f = float(rng.uniform(f_lo, f_hi))
        p = int(np.floor(f * t))
        lens.append((t, p, t - p))
    return rng, lens


def ragged_episodes(w: Workload, n: Optional[int] = None, scale_len: float = 1.0) -> List[Episode]:
    """The ragged batch: lengths first, then each episode's tensors in order.

    ``scale_len`` < 1 shrinks the length range (same recipe, smaller episodes)
    for fast checks; the full workload uses 1.0.
    """
    n = w.n_episodes if n is None else n
    lo, hi = int(4096 * scale_len), int(16384 * scale_len)
    rng, lens = draw_ragged_lengths(w.seed, n, lo, hi)
    return [draw_episode(rng, w.geometry, w.dtype, p, s, t) for (t, p, s) in lens]


def stack_inputs(w: Workload, t_total: Optional[int] = None, d_model: Optional[int] = None,
                 n_layers: Optional[int] = None):
    """Inputs of the stacked-layer workload, rounded to bf16 bits.

    Draw order: sanitized token states x0 [T, d_model], then an independent
    contaminated stream [T, d_model] (the contaminated run at crop point P is
    x0[:P] ++ contaminated[P:]), then per layer in order W_q [dm, Hq*d],
    W_k [dm, Hkv*d], W_v [dm, Hkv*d], W_o [Hq*d, dm], each N(0, 1/dm).
    """
    T = w.t_total if t_total is None else t_total
    dm = w.d_model if d_model is None else d_model
    L = w.n_layers if n_layers is None else n_layers
    g = w.geometry
    rng = np.random.default_rng(w.seed)
    x0 = f32_to_bf16_bits(_normal(rng, (T, dm)))
    xc = f32_to_bf16_bits(_normal(rng, (T, dm)))
    std = np.float32(1.0 / np.sqrt(dm))
    layers = []
    for _ in range(L):
        wq = f32_to_bf16_bits(_normal(rng, (dm, g.n_q_heads * g.head_dim)) * std)
        wk = f32_to_bf16_bits(_normal(rng, (dm, g.n_kv_heads * g.head_dim)) * std)
        wv = f32_to_bf16_bits(_normal(rng, (dm, g.n_kv_heads * g.head_dim)) * std)
        wo = f32_to_bf16_bits(_normal(rng, (g.n_q_heads * g.head_dim, dm)) * std)
        layers.append((wq, wk, wv, wo))
    return x0, xc, layers
