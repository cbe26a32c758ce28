"""Degenerate cases of the replay path on the device.

* The target enters at the first transition (tau = 1): the crop keeps nothing,
  the replay recomputes all T transitions (Corollary 1 with tau = 1) and equals
  the full reset bit for bit (Theorem 1).
* A sequence with an empty suffix inside a batch: it is skipped, its length is
  unchanged, and the other sequence's output is what it is alone.
* A call whose every suffix is empty: a no-op that counts no recomputed token.
"""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import assert_close, contaminated_then_crop, dev, make_pool, oracle_suffix

pytestmark = pytest.mark.gpu

SCALE = 128 ** -0.5
GEOM = W.AttnGeometry(32, 8, 128)


def _suffix(ep):
    return tuple(dev(getattr(ep, x)[ep.prefix:], ep.dtype) for x in ("q", "k", "v"))


def _whole(ep):
    return tuple(dev(getattr(ep, x), ep.dtype) for x in ("q", "k", "v"))


def test_target_in_first_transition_crops_to_zero():
    rng = np.random.default_rng(1)
    ep = W.draw_episode(rng, GEOM, "bf16", 0, 700, 500)
    pool = make_pool(GEOM, "bf16", 2 * 44 + 8, 2, 64)
    contaminated_then_crop(pool, ep, 0, SCALE)
    assert pool.seq_len(0) == 0
    before = pool.recomputed_tokens.value
    q, k, v = _suffix(ep)
    o = torch.empty_like(q)
    assert pool.replay(0, [0], [ep.suffix], q, k, v, o, SCALE) == 0
    assert pool.recomputed_tokens.value - before == ep.t_sanitized
    assert pool.seq_len(0) == ep.t_sanitized
    full = torch.empty_like(q)
    assert pool.full_reset(0, [1], [ep.t_sanitized], q, k, v, full, SCALE) == 0
    assert torch.equal(o, full)
    assert_close(o.float().cpu().numpy(), oracle_suffix(ep, SCALE), "bf16", "tau = 1")


def test_empty_suffix_in_a_batch_is_skipped():
    rng = np.random.default_rng(2)
    a = W.draw_episode(rng, GEOM, "bf16", 300, 0, 400)
    b = W.draw_episode(rng, GEOM, "bf16", 517, 250, 600)
    pool = make_pool(GEOM, "bf16", 3 * 48 + 8, 3, 64)
    contaminated_then_crop(pool, a, 0, SCALE)
    contaminated_then_crop(pool, b, 1, SCALE)
    q, k, v = _suffix(b)
    o = torch.empty_like(q)
    assert pool.replay(0, [0, 1], [0, b.suffix], q, k, v, o, SCALE) == 0
    assert pool.seq_len(0) == a.prefix
    assert pool.seq_len(1) == b.t_sanitized
    fq, fk, fv = _whole(b)
    full = torch.empty_like(fq)
    assert pool.full_reset(0, [2], [b.t_sanitized], fq, fk, fv, full, SCALE) == 0
    assert torch.equal(full[b.prefix:], o)
    assert_close(o.float().cpu().numpy(), oracle_suffix(b, SCALE), "bf16", "batch with an empty suffix")


def test_all_empty_call_is_a_no_op():
    rng = np.random.default_rng(3)
    ep = W.draw_episode(rng, GEOM, "bf16", 211, 64, 300)
    pool = make_pool(GEOM, "bf16", 2 * 20 + 8, 2, 32)
    contaminated_then_crop(pool, ep, 0, SCALE)
    st0 = pool.state()
    before = pool.recomputed_tokens.value
    zq = torch.empty((0, GEOM.n_q_heads, GEOM.head_dim), dtype=torch.bfloat16, device="cuda")
    zk = torch.empty((0, GEOM.n_kv_heads, GEOM.head_dim), dtype=torch.bfloat16, device="cuda")
    assert pool.replay(0, [0, 1], [0, 0], zq, zk, zk, torch.empty_like(zq), SCALE) == 0
    assert pool.recomputed_tokens.value == before
    st1 = pool.state()
    for key in st0:
        assert np.array_equal(np.asarray(st0[key]), np.asarray(st1[key])), key
