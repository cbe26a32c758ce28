"""Plain CPU oracle of deterministic seeded sampling.  TEST INFRASTRUCTURE ONLY.

Only ``tests/`` import this module; it shares no code with
``paper_2609_04875_amd``.

Theorem 1 needs decoding to be deterministic, or its randomness source fixed
(assumption A1); the paper samples at temperature 0.7 under matched seeds for
its token-for-token agreement test (Section 4).  Its sampler is not described,
so the readings are:

  S1 the next token of row i is argmax_v (l[i][v] / T + g[i][v]) (Gumbel-max:
     a draw from softmax(l / T)), with g = -log(-log(u)); at T = 0 it is
     argmax_v l[i][v]; ties go to the lowest index;
  S2 u[i][v] comes from the counter-based generator Philox4x64-10 (Salmon,
     Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
     SC 2011): one call with counter (v div 4, position_i, stream_i, 0) and key
     (seed, 0) gives four 64-bit words for v = 4 (v div 4) + 0..3; a word x maps
     to u = (floor(x / 2^41) + 1/2) / 2^23 = (2m + 1) / 2^24 with m < 2^23, a
     value in (0, 1) that fp32 holds exactly;
  S3 the argmax decides in fp32, the kernel's precision: g = -log(-log(u)) and
     l / T + g are formed in fp32.  The two sides' fp32 logarithms may differ
     in the last bit, so the oracle also reports each row's gap between its
     best and second-best fp32 score: a test can tell such a near-tie from a
     wrong pick.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np

MASK64 = (1 << 64) - 1
# Philox4x64 round multipliers and key increments (Weyl sequence), as published
M0, M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157
W0, W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B


def _mulhilo(a: int, b: int) -> Tuple[int, int]:
    p = a * b
    return p >> 64, p & MASK64


def philox4x64_10(counter: Sequence[int], key: Sequence[int]) -> Tuple[int, int, int, int]:
    """Ten rounds: each multiplies words 0 and 2 by M0, M1, mixes the high
    halves with words 1, 3 and the key, then bumps the key by (W0, W1)."""
    c0, c1, c2, c3 = (int(x) & MASK64 for x in counter)
    k0, k1 = (int(x) & MASK64 for x in key)
    for _ in range(10):
        hi0, lo0 = _mulhilo(M0, c0)
        hi1, lo1 = _mulhilo(M1, c2)
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0, k1 = (k0 + W0) & MASK64, (k1 + W1) & MASK64
    return c0, c1, c2, c3


def uniforms(vocab: int, position: int, stream: int, seed: int) -> np.ndarray:
    """u[v] for v < vocab (S2), as float64 holding fp32-exact values."""
    out = np.empty(vocab, dtype=np.float64)
    for b in range((vocab + 3) // 4):
        words = philox4x64_10((b, position, stream, 0), (seed, 0))
        for j, x in enumerate(words):
            v = 4 * b + j
            if v < vocab:
                out[v] = ((x >> 41) + 0.5) / float(1 << 23)
    return out


def sample(logits: np.ndarray, temperature: float, seed: int, streams: Sequence[int],
           positions: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Tokens per row (S1-S3) and each row's gap between its best and
    second-best fp32 score (0 at an exact tie)."""
    n, vocab = logits.shape
    tokens = np.empty(n, dtype=np.int64)
    gaps = np.empty(n, dtype=np.float64)
    t32 = np.float32(temperature)
    for i in range(n):
        l = logits[i].astype(np.float32)
        if temperature == 0:
            score = l
        else:
            u = uniforms(vocab, positions[i], streams[i], seed).astype(np.float32)
            g = -np.log(-np.log(u))                  # fp32 throughout
            score = (l / t32 + g).astype(np.float32)
        tokens[i] = int(np.argmax(score))            # first maximum: lowest index
        top2 = np.sort(score.astype(np.float64))[-2:] if vocab > 1 else np.array([-np.inf, score[0]])
        gaps[i] = top2[1] - top2[0]
    return tokens, gaps
