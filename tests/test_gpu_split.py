"""Split-key replay (partial softmax states per absolute key range, combined in
fixed order) against the fp64 oracle.  The split is taken when a launch would
leave CUs idle and the pool has a workspace; the result is the same softmax
attention (Section 3.2, replay by prefill), so the bf16 tolerance applies."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import (assert_close, contaminated_then_crop, dev, errors, log, make_pool,
                         oracle_suffix)

pytestmark = pytest.mark.gpu

GEOM = W.AttnGeometry(32, 8, 128)


def _blocks(n, B=16):
    return -(-n // B)


def _chunked(pool, ep, chunk, scale):
    outs = []
    for c0 in range(0, ep.suffix, chunk):
        n = min(chunk, ep.suffix - c0)
        sl = slice(ep.prefix + c0, ep.prefix + c0 + n)
        q, k, v = (dev(getattr(ep, x)[sl], "bf16") for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, [0], [n], q, k, v, o, scale) == 0
        outs.append(o)
    return torch.cat(outs)


@pytest.mark.parametrize("P,S,C", [(4000, 512, 128), (1500, 200, 37), (63, 64, 64)])
def test_split_chunked_replay_matches_oracle(P, S, C):
    log(f"split chunked P={P} S={S} C={C}")
    rng = np.random.default_rng(P + S)
    ep = W.draw_episode(rng, GEOM, "bf16", P, S, P + 40)
    scale = 128 ** -0.5
    nb = _blocks(P + S + 40) + _blocks(P + S) + 4
    split = make_pool(GEOM, "bf16", nb, 1, 512, split_q=C)
    plain = make_pool(GEOM, "bf16", nb, 1, 512)
    outs = []
    for pool in (split, plain):
        contaminated_then_crop(pool, ep, 0, scale)
        outs.append(_chunked(pool, ep, C, scale))
    ref = oracle_suffix(ep, scale)
    assert_close(outs[0].float().cpu().numpy(), ref, "bf16", "split")
    assert_close(outs[1].float().cpu().numpy(), ref, "bf16", "plain")
    # the split path really split (else this test would not cover it)
    assert not torch.equal(outs[0], outs[1])


def test_split_replay_is_deterministic():
    rng = np.random.default_rng(31)
    ep = W.draw_episode(rng, GEOM, "bf16", 3000, 256, 3100)
    scale = 128 ** -0.5
    pool = make_pool(GEOM, "bf16", 2 * _blocks(3300) + 4, 1, 512, split_q=256)
    contaminated_then_crop(pool, ep, 0, scale)
    q, k, v = (dev(getattr(ep, x)[ep.prefix:], "bf16") for x in ("q", "k", "v"))
    o1, o2 = torch.empty_like(q), torch.empty_like(q)
    assert pool.replay(0, [0], [ep.suffix], q, k, v, o1, scale, commit=False) == 0
    assert pool.replay(0, [0], [ep.suffix], q, k, v, o2, scale, commit=False) == 0
    assert torch.equal(o1, o2)
    assert_close(o1.float().cpu().numpy(), oracle_suffix(ep, scale), "bf16", "split one-shot")


def test_split_varlen_small_batch():
    # few short suffixes against long prefixes: a launch with few workgroups
    rng = np.random.default_rng(32)
    eps = [W.draw_episode(rng, GEOM, "bf16", p, s, p + s) for p, s in ((2000, 17), (777, 40), (3100, 5))]
    scale = 128 ** -0.5
    nb = sum(2 * _blocks(e.t_sanitized) for e in eps) + 8
    pool = make_pool(GEOM, "bf16", nb, 3, 512, split_q=sum(e.suffix for e in eps))
    for i, ep in enumerate(eps):
        contaminated_then_crop(pool, ep, i, scale)
    q = torch.cat([dev(e.q[e.prefix:], "bf16") for e in eps])
    k = torch.cat([dev(e.k[e.prefix:], "bf16") for e in eps])
    v = torch.cat([dev(e.v[e.prefix:], "bf16") for e in eps])
    o = torch.empty_like(q)
    assert pool.replay(0, [0, 1, 2], [e.suffix for e in eps], q, k, v, o, scale) == 0
    got = o.float().cpu().numpy()
    off = 0
    for i, ep in enumerate(eps):
        assert_close(got[off:off + ep.suffix], oracle_suffix(ep, scale), "bf16", f"episode {i}")
        off += ep.suffix


def test_long_horizon_split_full_size_sampled():
    w = W.workload("long32k_chunk512_llama8b_bf16")
    log(f"workload {w.name} with split-key chunks")
    ep = W.single_episode(w)
    pool = make_pool(w.geometry, "bf16", _blocks(36864) + 8, 1, 2400, split_q=w.chunk)
    contaminated_then_crop(pool, ep, 0, w.scale)
    o = _chunked(pool, ep, w.chunk, w.scale)
    # every chunk's first two and last two tokens and 96 random ones, all 32
    # query heads of each (4096 of the 131,072 output rows)
    rng = np.random.default_rng(7)
    edges = [c + x for c in range(0, 4096, w.chunk) for x in (0, 1, w.chunk - 2, w.chunk - 1)]
    rest = np.setdiff1d(np.arange(4096), edges)
    toks = np.sort(np.concatenate([edges, rng.choice(rest, 96, replace=False)]))
    rows = (toks[:, None] * 32 + np.arange(32)[None, :]).reshape(-1)
    log(f"oracle on {rows.size} rows ({toks.size} tokens x 32 heads)")
    ref = oracle_suffix(ep, w.scale, rows=rows)
    assert_close(o.float().cpu().numpy().reshape(-1, 128)[rows], ref, "bf16", w.name)


@pytest.mark.parametrize("geom,P,S", [(W.AttnGeometry(8, 8, 64), 512, 128), (W.AttnGeometry(4, 2, 128), 301, 70),
                                      (W.AttnGeometry(8, 8, 64), 0, 100)])
def test_fp32_split_replay_matches_oracle(geom, P, S):
    """fp32 pools split keys too when a call launches few workgroups (the tiny
    workload: 2 query tiles x 8 heads); partials merge into fp32 output within
    the fp32 tolerance."""
    log(f"fp32 split {geom} P={P} S={S}")
    rng = np.random.default_rng(P + 7 * S)
    ep = W.draw_episode(rng, geom, "f32", P, S, P + 33)
    scale = geom.head_dim ** -0.5
    nb = _blocks(P + S + 33) + _blocks(P + S) + 4
    outs = []
    for split_q in (S, 0):
        pool = make_pool(geom, "f32", nb, 1, 64, split_q=split_q)
        contaminated_then_crop(pool, ep, 0, scale, poison=True)
        q, k, v = (dev(getattr(ep, x)[ep.prefix:], "f32") for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, [0], [S], q, k, v, o, scale) == 0
        outs.append(o)
    ref = oracle_suffix(ep, scale)
    assert_close(outs[0].cpu().numpy(), ref, "f32", "split")
    assert_close(outs[1].cpu().numpy(), ref, "f32", "plain")
    assert not torch.equal(outs[0], outs[1])
