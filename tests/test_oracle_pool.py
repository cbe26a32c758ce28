"""Pins of the oracle's paged-pool semantics (restore = crop, Section 3.4 (b);
Algorithm 1 restore and replay steps; Lemma 1; Theorem 1; Corollary 1).

Pinned by a hand-worked trace (tests/golden/pool_worked_example.json),
exhaustive invariants on tiny pools, an independent token-at-a-time allocator,
and the paper's theorems stated as properties.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import PoolModel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _apply(pool, step):
    if step["op"] == "crop":
        return pool.crop(step["seqs"], step["lens"])
    rc = pool.reserve(step["seqs"], step["lens"])
    if rc == 0 and step.get("commit"):
        pool.commit(step["seqs"], step["lens"])
    return rc


def _run_trace(spec):
    pool = PoolModel(spec["n_blocks"], spec["max_seqs"], spec["max_blocks"], spec["block_size"],
                     spec["init_free_order"])
    for i, step in enumerate(spec["steps"]):
        rc = _apply(pool, step)
        assert rc == step["status"], f"step {i}"
        np.testing.assert_array_equal(pool.tables, np.array(step["tables"]), err_msg=f"step {i}")
        np.testing.assert_array_equal(pool.lens, np.array(step["seq_lens"]), err_msg=f"step {i}")
        np.testing.assert_array_equal(pool.free, np.array(step["free"]), err_msg=f"step {i}")
        assert pool.top == step["top"], f"step {i}"


def test_hand_worked_trace():
    with open(os.path.join(GOLDEN, "pool_worked_example.json")) as f:
        spec = json.load(f)
    _run_trace(spec)
    _run_trace(spec["permuted"])


def _invariants(pool, n_seqs):
    held = []
    for s in range(n_seqs):
        n = int(pool.nalloc[s])
        row = pool.tables[s]
        assert (row[:n] >= 0).all() and (row[n:] == -1).all()
        assert n >= math.ceil(int(pool.lens[s]) / pool.B)
        held.extend(row[:n].tolist())
    free = pool.free[: pool.top].tolist()
    # conservation and no duplicates: held + free is exactly the id set
    assert len(held) + pool.top == pool.n_blocks
    assert sorted(held + free) == list(range(pool.n_blocks))


@pytest.mark.parametrize("B", [1, 4, 16])
def test_exhaustive_single_sequence_crop(B):
    max_len = 64
    nb = math.ceil(max_len / B)
    for length in range(0, max_len + 1):
        for L in range(0, length + 1):
            pool = PoolModel(nb, 1, nb, B)
            assert pool.reserve([0], [length]) == 0
            pool.commit([0], [length])
            before = pool.tables[0].copy()
            top0 = pool.top
            assert pool.crop([0], [L]) == 0
            keep, had = math.ceil(L / B), math.ceil(length / B)
            np.testing.assert_array_equal(pool.tables[0][:keep], before[:keep])   # kept prefix unchanged
            assert (pool.tables[0][keep:] == -1).all()
            # freed = exactly the removed tail, pushed in ascending logical order
            np.testing.assert_array_equal(pool.free[top0: pool.top], before[keep:had])
            assert pool.lens[0] == L
            _invariants(pool, 1)


def test_exhaustive_multi_sequence_crop_order():
    B, nb = 4, 48
    rng = np.random.default_rng(0)
    for n_seqs in (2, 3):
        for _ in range(60):
            lens = rng.integers(0, 33, size=n_seqs).tolist()
            pool = PoolModel(nb, n_seqs, 9, B, init_free_order=rng.permutation(nb).tolist())
            assert pool.reserve(list(range(n_seqs)), lens) == 0
            pool.commit(list(range(n_seqs)), lens)
            order = rng.permutation(n_seqs).tolist()
            new = [int(rng.integers(0, lens[s] + 1)) for s in order]
            rows = pool.tables.copy()
            top0 = pool.top
            assert pool.crop(order, new) == 0
            expect = []
            for s, L in zip(order, new):
                expect.extend(rows[s][math.ceil(L / B): math.ceil(lens[s] / B)].tolist())
            np.testing.assert_array_equal(pool.free[top0: pool.top], expect)
            _invariants(pool, n_seqs)


def _token_at_a_time(n_blocks, B, max_blocks, n_seqs, calls, init):
    """Independent allocator: one token at a time; a block is popped exactly when a
    token lands on the first slot of a block.  ``calls`` is a list of
    (seq, n_tokens) served in order."""
    free = list(init) if init is not None else list(range(n_blocks - 1, -1, -1))
    tables = [[-1] * max_blocks for _ in range(n_seqs)]
    pos = [0] * n_seqs
    for s, n in calls:
        for _ in range(n):
            if pos[s] % B == 0:
                tables[s][pos[s] // B] = free.pop()
            pos[s] += 1
    return np.array(tables, np.int32), free


@pytest.mark.parametrize("B", [1, 3, 16])
def test_batched_reserve_equals_token_at_a_time(B):
    rng = np.random.default_rng(B)
    for _ in range(40):
        lens = rng.integers(0, 70, size=3).tolist()
        nb = sum(math.ceil(x / B) for x in lens) + 5
        init = rng.permutation(nb).tolist()
        pool = PoolModel(nb, 3, 80, B, init_free_order=init)
        cut = [int(rng.integers(0, x + 1)) for x in lens]
        rest = [a - c for a, c in zip(lens, cut)]
        order1, order2 = rng.permutation(3).tolist(), rng.permutation(3).tolist()
        assert pool.reserve(order1, [cut[s] for s in order1]) == 0
        pool.commit(order1, [cut[s] for s in order1])
        assert pool.reserve(order2, [rest[s] for s in order2]) == 0
        pool.commit(order2, [rest[s] for s in order2])
        calls = [(s, cut[s]) for s in order1] + [(s, rest[s]) for s in order2]
        t_tables, t_free = _token_at_a_time(nb, B, 80, 3, calls, init)
        np.testing.assert_array_equal(pool.tables, t_tables)
        assert pool.top == len(t_free)
        np.testing.assert_array_equal(pool.free[: pool.top], t_free)
        _invariants(pool, 3)


def test_crop_then_reappend_reverses_the_freed_tail():
    # LIFO consequence: ids freed in ascending order come back in descending order.
    pool = PoolModel(16, 1, 16, 4)
    pool.reserve([0], [40]); pool.commit([0], [40])
    row = pool.tables[0].copy()
    pool.crop([0], [12])
    pool.reserve([0], [28]); pool.commit([0], [28])
    np.testing.assert_array_equal(pool.tables[0][:3], row[:3])
    np.testing.assert_array_equal(pool.tables[0][3:10], row[3:10][::-1])


@pytest.mark.parametrize("bad", ["dup", "range", "neg", "seq", "nomem", "width"])
def test_errors_change_nothing(bad):
    pool = PoolModel(7, 3, 4, 4)     # 5 of 7 blocks in use after this
    pool.reserve([0, 1], [9, 5]); pool.commit([0, 1], [9, 5])
    snap = pool.state()
    if bad == "dup":
        assert pool.crop([1, 1], [0, 0]) == oracle.EINVAL
    elif bad == "range":
        assert pool.crop([0, 1], [3, 6]) == oracle.ERANGE
    elif bad == "neg":
        assert pool.crop([0], [-1]) == oracle.ERANGE
    elif bad == "seq":
        assert pool.crop([3], [0]) == oracle.EINVAL
    elif bad == "nomem":
        assert pool.reserve([2, 0], [8, 7]) == oracle.ENOMEM
    elif bad == "width":
        assert pool.reserve([1], [12]) == oracle.ERANGE
    after = pool.state()
    for key in snap:
        np.testing.assert_array_equal(snap[key], after[key])


# --------------------------------------------------------------------------- #
# the paper's statements as properties of the oracle                           #
# --------------------------------------------------------------------------- #
def _episode(rng, P, S_contam, S_san, hq=4, hkv=2, d=8):
    T = P + S_san
    q, k, v = rng.standard_normal((T, hq, d)), rng.standard_normal((T, hkv, d)), rng.standard_normal((T, hkv, d))
    cq, ck, cv = (rng.standard_normal((S_contam, h, d)) for h in (hq, hkv, hkv))
    return q, k, v, cq, ck, cv


@pytest.mark.parametrize("P,Sc,Ss,B", [(13, 9, 7, 4), (16, 4, 4, 4), (5, 20, 1, 16), (0, 6, 6, 4)])
def test_lemma1_theorem1_on_the_oracle_pool(P, Sc, Ss, B):
    rng = np.random.default_rng(P * 100 + Sc)
    q, k, v, cq, ck, cv = _episode(rng, P, Sc, Ss)
    scale = 0.35
    nb = 64
    pool = PoolModel(nb, 2, 16, B, init_free_order=rng.permutation(nb).tolist(),
                     n_layers=1, n_kv_heads=2, head_dim=8)
    # contaminated run: shared prefix, then the contaminated suffix
    contaminated = [np.concatenate([a[:P], c]) for a, c in ((q, cq), (k, ck), (v, cv))]
    oracle.prefill(pool, 0, [0], [P + Sc], *contaminated, scale)
    kept_k = pool.gather(0, 0, P)[0].copy()
    # restore = crop to tau - 1 = P, then replay the sanitized suffix
    assert pool.crop([0], [P]) == 0
    out = oracle.prefill(pool, 0, [0], [Ss], q[P:], k[P:], v[P:], scale)[0]
    # Lemma 1: the kept prefix is untouched
    np.testing.assert_array_equal(pool.gather(0, 0, P)[0], kept_k)
    # Theorem 1: equals the full reset (B5) on the sanitized trajectory, rows P..T-1
    ref_pool = PoolModel(nb, 1, 16, B, n_layers=1, n_kv_heads=2, head_dim=8)
    full = oracle.prefill(ref_pool, 0, [0], [P + Ss], q, k, v, scale)[0]
    np.testing.assert_array_equal(out, full[P:])
    # the logical caches agree
    np.testing.assert_array_equal(pool.gather(0, 0, P + Ss)[0], ref_pool.gather(0, 0, P + Ss)[0])
    # Corollary 1: the replay ran F on exactly T - tau + 1 = Ss tokens
    assert oracle.recomputed_transitions(P + Ss, P + 1) == Ss


def test_any_earlier_clean_boundary_is_equally_exact():
    # Theorem 1 holds from any earlier clean boundary c < tau - 1; it costs T - c.
    rng = np.random.default_rng(5)
    P, Sc, Ss, B = 21, 6, 5, 4
    q, k, v, cq, ck, cv = _episode(rng, P, Sc, Ss)
    contaminated = [np.concatenate([a[:P], c]) for a, c in ((q, cq), (k, ck), (v, cv))]
    outs = []
    for c in (0, (P // B) * B, P - 3, P):
        pool = PoolModel(40, 1, 16, B, n_layers=1, n_kv_heads=2, head_dim=8)
        oracle.prefill(pool, 0, [0], [P + Sc], *contaminated, 0.3)
        assert pool.crop([0], [c]) == 0
        out = oracle.prefill(pool, 0, [0], [P + Ss - c], q[c:], k[c:], v[c:], 0.3)[0]
        outs.append(out[P - c:])
        assert out.shape[0] == oracle.recomputed_transitions(P + Ss, c + 1)
    for o in outs[1:]:
        np.testing.assert_array_equal(o, outs[0])


def test_negative_controls_differ_from_full_reset():
    # B0 (no crop) and span-only excision keep KV computed after the target:
    # both must differ from the counterfactual by far more than any tolerance.
    rng = np.random.default_rng(6)
    P, Sc, Ss = 24, 8, 8
    q, k, v, cq, ck, cv = _episode(rng, P, Sc, Ss)
    full = oracle.attention(q, k, v, 0, 0.5)[P:]
    # no crop: the replay is appended after the contaminated suffix
    kk = np.concatenate([k[:P], ck, k[P:]]); vv = np.concatenate([v[:P], cv, v[P:]])
    no_crop = oracle.attention(q[P:], kk, vv, P + Sc, 0.5)
    assert np.abs(no_crop - full).max() > 0.05
    # span-only excision: drop the target's first 3 slots, keep the rest of the
    # contaminated suffix as the "replayed" state
    kk = np.concatenate([k[:P], ck[3:]]); vv = np.concatenate([v[:P], cv[3:]])
    n = Sc - 3
    span = oracle.attention(cq[3:], kk, vv, P, 0.5)
    assert np.abs(span[:n] - full[:n]).max() > 0.05


def test_corollary1_closed_forms():
    with open(os.path.join(GOLDEN, "corollary1_counts.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        assert oracle.recomputed_transitions(c["T"], c["tau"]) == c["recomputed"], c["name"]
        assert oracle.replay_gain(c["T"], c["tau"]) == pytest.approx(c["gain"], rel=1e-15), c["name"]
