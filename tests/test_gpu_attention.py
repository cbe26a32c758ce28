"""GPU parity of the replay prefill against the fp64 oracle, and the paper's
statements checked on the device: selective replay equals the full reset
(Theorem 1, bitwise here), replay from an earlier clean boundary is equally
exact (Theorem 1 / checkpoint granularity, Section 4), the recompute count is
T - tau + 1 (Corollary 1), runs are deterministic (assumption A1), chunked
replay equals one-shot, and the negative controls (no crop) fail."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import (assert_close, bits, contaminated_then_crop, dev, errors, log, make_pool,
                         oracle_suffix, storage_f64)

pytestmark = pytest.mark.gpu


def _replay(pool, ep, seq, scale, commit=True):
    q, k, v = (dev(getattr(ep, x)[ep.prefix:], ep.dtype) for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    assert pool.replay(0, [seq], [ep.suffix], q, k, v, o, scale, commit=commit) == 0
    return o


def _full_reset(pool, ep, seq, scale):
    q, k, v = (dev(getattr(ep, x), ep.dtype) for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    assert pool.full_reset(0, [seq], [ep.t_sanitized], q, k, v, o, scale) == 0
    return o


def _blocks(n, B=16):
    return -(-n // B)


def test_tiny_fp32_episode():
    w = W.workload("tiny_mha8_d64_p512_s128_f32")
    log(f"workload {w.name}")
    ep = W.single_episode(w)
    pool = make_pool(w.geometry, "f32", 2 * _blocks(640) + 4, 2, 64)
    co = contaminated_then_crop(pool, ep, 0, w.scale)
    o = _replay(pool, ep, 0, w.scale)
    assert pool.recomputed_tokens.value == 640 + 128          # contaminated run + replay
    ref = oracle_suffix(ep, w.scale)
    assert_close(o.cpu().numpy(), ref, "f32", w.name)
    # Theorem 1: equals the full reset of the sanitized 640 tokens, bitwise
    full = _full_reset(pool, ep, 1, w.scale)
    assert torch.equal(full[ep.prefix:], o)
    # Lemma 1: the full reset's rows before tau equal the contaminated run's
    assert torch.equal(full[: ep.prefix], co[: ep.prefix])


GEOMS = [
    # (Hq, Hkv, d, P, S)
    (32, 8, 128, 300, 77),
    (32, 8, 128, 0, 130),
    (32, 8, 128, 1021, 1),
    (8, 8, 64, 129, 50),
    (64, 8, 128, 100, 33),
    (16, 2, 128, 47, 200),
    (4, 4, 128, 64, 64),
    # groups that do not divide 32: padded rows in every wave
    (28, 4, 128, 333, 101),      # the Qwen2.5-7B geometry, G = 7
    (24, 8, 128, 95, 60),        # G = 3
    (20, 4, 64, 17, 41),         # G = 5, d = 64
]


@pytest.mark.parametrize("hq,hkv,d,P,S", GEOMS)
def test_bf16_replay_matches_oracle(hq, hkv, d, P, S):
    geom = W.AttnGeometry(hq, hkv, d)
    log(f"bf16 geometry {hq}/{hkv}/{d} P={P} S={S}")
    rng = np.random.default_rng(hq * 1000 + P)
    ep = W.draw_episode(rng, geom, "bf16", P, S, P + S + 5)
    scale = d ** -0.5
    pool = make_pool(geom, "bf16", _blocks(P + S + 5) + _blocks(P + S) + 2, 1, 128)
    contaminated_then_crop(pool, ep, 0, scale)
    o = _replay(pool, ep, 0, scale)
    assert_close(o.float().cpu().numpy(), oracle_suffix(ep, scale), "bf16", f"{hq}/{hkv}/{d}")


def test_bf16_selective_equals_full_reset_bitwise_and_deterministic():
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(21)
    ep = W.draw_episode(rng, geom, "bf16", 757, 300, 1100)
    scale = 128 ** -0.5
    pool = make_pool(geom, "bf16", 3 * _blocks(1100) + 8, 3, 128)
    contaminated_then_crop(pool, ep, 0, scale)
    o1 = _replay(pool, ep, 0, scale, commit=False)
    o2 = _replay(pool, ep, 0, scale, commit=False)
    assert torch.equal(o1, o2)                                  # (A1) determinism
    full = _full_reset(pool, ep, 1, scale)
    assert torch.equal(full[ep.prefix:], o1)                    # Theorem 1, bitwise


def test_group7_selective_equals_full_reset_bitwise():
    """Theorem 1 at G = 7 (28 query / 4 KV heads): the padded rows change nothing."""
    geom = W.AttnGeometry(28, 4, 128)
    rng = np.random.default_rng(77)
    ep = W.draw_episode(rng, geom, "bf16", 1003, 250, 1300)
    scale = 128 ** -0.5
    pool = make_pool(geom, "bf16", 2 * _blocks(1300) + 8, 2, 128)
    contaminated_then_crop(pool, ep, 0, scale)
    o = _replay(pool, ep, 0, scale, commit=False)
    full = _full_reset(pool, ep, 1, scale)
    assert torch.equal(full[ep.prefix:], o)
    assert_close(o.float().cpu().numpy(), oracle_suffix(ep, scale), "bf16", "G=7")


def test_earlier_clean_boundary_is_equally_exact():
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(22)
    P, S = 421, 90
    ep = W.draw_episode(rng, geom, "bf16", P, S, P + 60)
    scale = 128 ** -0.5
    outs = []
    for c in (0, (P // 16) * 16, P - 5, P):
        pool = make_pool(geom, "bf16", 2 * _blocks(P + S + 60) + 4, 1, 128)
        contaminated_then_crop(pool, ep, 0, scale)
        assert pool.crop([0], [c]) == 0
        q, k, v = (dev(getattr(ep, x)[c:], "bf16") for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        before = pool.recomputed_tokens.value
        assert pool.replay(0, [0], [P + S - c], q, k, v, o, scale) == 0
        assert pool.recomputed_tokens.value - before == oracle.recomputed_transitions(P + S, c + 1)
        outs.append(o[P - c:])
    for o in outs[1:]:
        assert torch.equal(o, outs[0])


def test_chunked_replay_equals_one_shot():
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(23)
    P, S, C = 900, 384, 96
    ep = W.draw_episode(rng, geom, "bf16", P, S, P + 50)
    scale = 128 ** -0.5
    pool = make_pool(geom, "bf16", 3 * _blocks(P + S + 50) + 4, 2, 128)
    contaminated_then_crop(pool, ep, 0, scale)
    one = _replay(pool, ep, 0, scale, commit=False)
    outs = []
    for c0 in range(0, S, C):
        q, k, v = (dev(getattr(ep, x)[P + c0:P + c0 + C], "bf16") for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, [0], [C], q, k, v, o, scale) == 0
        outs.append(o)
    assert torch.equal(torch.cat(outs), one)
    assert pool.seq_len(0) == P + S


def test_negative_control_without_crop_differs():
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(24)
    ep = W.draw_episode(rng, geom, "bf16", 500, 120, 700)
    scale = 128 ** -0.5
    pool = make_pool(geom, "bf16", 3 * _blocks(820) + 4, 1, 128)
    cq, ck, cv = (dev(ep.contaminated(x), "bf16") for x in ("q", "k", "v"))
    co = torch.empty_like(cq)
    assert pool.replay(0, [0], [700], cq, ck, cv, co, scale) == 0
    # B0-like: replay appended after the contaminated suffix, no crop
    o = _replay(pool, ep, 0, scale)
    mx, rel = errors(o.float().cpu().numpy(), oracle_suffix(ep, scale))
    assert mx > 0.2 and rel > 0.1, (mx, rel)


def test_negative_control_span_only_excision_differs():
    """The span-only invalidation boundary of the ablation (Section 4, Table 4):
    cut the target's own slots out of the contaminated cache but keep the KV of
    everything computed after it.  On the GPU the kept state is the prefix
    followed by the contaminated suffix past the target span; its outputs must
    differ from the full reset of the sanitized trajectory by far more than the
    tolerance (the comparison has power), while matching the oracle for that
    same (wrong) state."""
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(25)
    P, S, Tc, z = 500, 120, 700, 3                 # the target: the first 3 contaminated tokens
    ep = W.draw_episode(rng, geom, "bf16", P, S, Tc)
    scale = 128 ** -0.5
    pool = make_pool(geom, "bf16", 2 * _blocks(Tc) + 8, 2, 128)
    span = {x: np.concatenate([getattr(ep, x)[:P], getattr(ep, "c" + x)[z:]]) for x in ("q", "k", "v")}
    sq, sk, sv = (dev(span[x], "bf16") for x in ("q", "k", "v"))
    so = torch.empty_like(sq)
    assert pool.replay(0, [0], [Tc - z], sq, sk, sv, so, scale) == 0
    full = _full_reset(pool, ep, 1, scale)
    n = min(S, Tc - P - z)
    mx, rel = errors(so[P:P + n].float().cpu().numpy(), full[P:P + n].float().cpu().numpy().astype(np.float64))
    log(f"span-only excision vs full reset: max|d| {mx:.3f}, rel {rel:.3f}")
    assert mx > 0.2 and rel > 0.1, (mx, rel)
    ref = oracle.attention(*(storage_f64(span[x][P:] if x == "q" else span[x], "bf16") for x in ("q", "k", "v")),
                           P, scale)
    assert_close(so[P:].float().cpu().numpy(), ref, "bf16", "span-only state")


def test_varlen_ragged_batch_reduced_lengths():
    w = W.workload("ragged16_llama8b_bf16")
    eps = W.ragged_episodes(w, scale_len=1 / 16)
    log("ragged: " + ", ".join(f"({e.prefix},{e.suffix})" for e in eps))
    n = len(eps)
    tot_blocks = sum(_blocks(e.t_contaminated) + _blocks(e.t_sanitized) for e in eps)
    pool = make_pool(w.geometry, "bf16", tot_blocks + 8, n, 128)
    for i, ep in enumerate(eps):
        contaminated_then_crop(pool, ep, i, w.scale)
    order = list(range(n))[::-1]                 # packed in a different order than ids
    q = torch.cat([dev(eps[i].q[eps[i].prefix:], "bf16") for i in order])
    k = torch.cat([dev(eps[i].k[eps[i].prefix:], "bf16") for i in order])
    v = torch.cat([dev(eps[i].v[eps[i].prefix:], "bf16") for i in order])
    o = torch.empty_like(q)
    before = pool.recomputed_tokens.value
    assert pool.replay(0, order, [eps[i].suffix for i in order], q, k, v, o, w.scale) == 0
    assert pool.recomputed_tokens.value - before == sum(e.suffix for e in eps)
    got = o.float().cpu().numpy()
    off = 0
    for i in order:
        ep = eps[i]
        assert_close(got[off:off + ep.suffix], oracle_suffix(ep, w.scale), "bf16", f"episode {i}")
        off += ep.suffix


def _sample_rows(rng, S, hq, n):
    toks = np.unique(np.concatenate([np.arange(min(4, S)), np.arange(max(0, S - 4), S),
                                     rng.integers(0, S, size=n)]))
    heads = rng.integers(0, hq, size=toks.shape[0])
    rows = np.concatenate([toks * hq + heads, toks * hq + (heads + hq // 2) % hq])
    return np.unique(rows)


def test_llama8b_workload_full_size_every_row():
    """8B geometry at its real shape: crop at 8189 (13 valid slots in the tail
    block), replay 2048; every one of the 2048 x 32 output rows against the
    oracle, with the bf16 acceptance metric (max |d| and sum|d| / sum|ref|)
    taken over the whole output, and every row against the GPU full reset of
    10237 tokens (bitwise)."""
    w = W.workload("llama8b_p8189_s2048_bf16")
    log(f"workload {w.name}")
    ep = W.single_episode(w)
    pool = make_pool(w.geometry, "bf16", _blocks(10240) + _blocks(10237) + 8, 2, 1024)
    contaminated_then_crop(pool, ep, 0, w.scale)
    assert pool.seq_len(0) == 8189
    o = _replay(pool, ep, 0, w.scale)
    assert pool.seq_len(0) == 10237
    got = o.float().cpu().numpy()
    log(f"{w.name}: oracle on all {ep.suffix} x 32 rows")
    ref = oracle_suffix(ep, w.scale)
    mx, rel = errors(got, ref)
    log(f"{w.name}: whole output max|d| {mx:.3e}, sum|d|/sum|ref| {rel:.3e}")
    assert_close(got, ref, "bf16", w.name)
    full = _full_reset(pool, ep, 1, w.scale)
    assert torch.equal(full[ep.prefix:], o)


def _ragged_tokens(rng, P, S, tile=64):
    """Suffix tokens to check in one episode: the first and last, the tokens
    on both sides of every query-tile edge near the ends, those whose absolute
    position straddles a 64-key tile edge (first and last such), and 32 at
    random."""
    t = [0, 1, tile - 1, tile, S - tile - 1, S - tile, S - 2, S - 1]
    first_edge = (-P) % tile                       # (P + t) % 64 == 0
    t += [first_edge - 1, first_edge, first_edge + tile - 1]
    last_edge = first_edge + ((S - 1 - first_edge) // tile) * tile
    t += [last_edge - 1, last_edge]
    t += rng.integers(0, S, size=32).tolist()
    return np.unique(np.clip(np.asarray(t), 0, S - 1))


def test_ragged_workload_full_size_sampled():
    """The 16-episode ragged batch at its configured lengths (T in [4096, 16384],
    about 82k suffix tokens) in one varlen launch; in every episode the first,
    last, tile-edge and diagonal-straddling tokens plus 32 random ones, all 32
    heads, against the oracle."""
    w = W.workload("ragged16_llama8b_bf16")
    log(f"workload {w.name}: drawing 16 episodes")
    eps = W.ragged_episodes(w)
    n = len(eps)
    log("ragged: " + ", ".join(f"({e.prefix},{e.suffix})" for e in eps))
    tot_blocks = sum(_blocks(e.t_contaminated) + _blocks(e.t_sanitized) for e in eps)
    pool = make_pool(w.geometry, "bf16", tot_blocks + 8, n, 1100)
    for i, ep in enumerate(eps):
        contaminated_then_crop(pool, ep, i, w.scale)
    order = list(range(n))[::-1]
    q = torch.cat([dev(eps[i].q[eps[i].prefix:], "bf16") for i in order])
    k = torch.cat([dev(eps[i].k[eps[i].prefix:], "bf16") for i in order])
    v = torch.cat([dev(eps[i].v[eps[i].prefix:], "bf16") for i in order])
    o = torch.empty_like(q)
    before = pool.recomputed_tokens.value
    assert pool.replay(0, order, [eps[i].suffix for i in order], q, k, v, o, w.scale) == 0
    assert pool.recomputed_tokens.value - before == sum(e.suffix for e in eps)
    got = o.float().cpu().numpy().reshape(-1, 32, 128)
    del q, k, v, o
    rng = np.random.default_rng(8)
    off = 0
    all_got, all_ref = [], []
    for i in order:
        ep = eps[i]
        toks = _ragged_tokens(rng, ep.prefix, ep.suffix)
        rows = (toks[:, None] * 32 + np.arange(32)[None, :]).reshape(-1)
        ref = oracle_suffix(ep, w.scale, rows=rows)
        g = got[off:off + ep.suffix].reshape(-1, 128)[rows]
        assert_close(g, ref, "bf16", f"episode {i} (P={ep.prefix}, S={ep.suffix})")
        all_got.append(g)
        all_ref.append(ref)
        off += ep.suffix
    mx, rel = errors(np.concatenate(all_got), np.concatenate(all_ref))
    log(f"{w.name}: {sum(x.shape[0] for x in all_got)} rows, max|d| {mx:.3e}, rel {rel:.3e}")


def test_long_horizon_chunked_full_size_sampled():
    """32768-token prefix, 4096-token suffix replayed in 512-token chunks."""
    w = W.workload("long32k_chunk512_llama8b_bf16")
    log(f"workload {w.name}")
    ep = W.single_episode(w)
    pool = make_pool(w.geometry, "bf16", _blocks(36864) + 8, 1, 2400)
    contaminated_then_crop(pool, ep, 0, w.scale)
    outs = []
    for c0 in range(0, ep.suffix, w.chunk):
        sl = slice(ep.prefix + c0, ep.prefix + c0 + w.chunk)
        q, k, v = (dev(getattr(ep, x)[sl], "bf16") for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, [0], [w.chunk], q, k, v, o, w.scale) == 0
        outs.append(o)
    o = torch.cat(outs)
    rng = np.random.default_rng(6)
    rows = _sample_rows(rng, ep.suffix, 32, 48)
    ref = oracle_suffix(ep, w.scale, rows=rows)
    assert_close(o.float().cpu().numpy().reshape(-1, 128)[rows], ref, "bf16", w.name)
