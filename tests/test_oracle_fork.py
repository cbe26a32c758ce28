"""Pins of the copy-on-write fork in the oracle pool (reading R5): a
hand-worked trace, and brute-force isolation under random forks, crops and
appends (every sequence reads back exactly the tokens written to it, and the
block counts equal the table entries naming each block)."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import EINVAL, OK, PoolModel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fork_worked_example.json")


def _apply(pool, st):
    if st["op"] == "append":
        assert pool.reserve(st["seqs"], st["q_lens"]) == OK
        pool.commit(st["seqs"], st["q_lens"])
    elif st["op"] == "fork":
        assert pool.fork(st["srcs"], st["dsts"]) == OK
    else:
        assert pool.crop(st["seqs"], st["new_lens"]) == OK


def test_fork_worked_example():
    with open(GOLDEN) as f:
        gd = json.load(f)
    pool = PoolModel(gd["n_blocks"], gd["max_seqs"], gd["max_blocks"], gd["B"])
    for st in gd["steps"]:
        top_before = pool.top
        _apply(pool, st)
        assert pool.tables.tolist() == st["tables"], st["op"]
        assert pool.lens.tolist() == st["lens"] and pool.top == st["top"] and pool.refs.tolist() == st["refs"]
        if "free_top_entries" in st:
            assert pool.free[top_before:pool.top].tolist() == st["free_top_entries"]
    assert pool.free.tolist() == gd["final_free"]


def _invariants(pool):
    counts = np.zeros(pool.n_blocks, np.int64)
    for s in range(pool.tables.shape[0]):
        row = pool.tables[s, :pool.nalloc[s]]
        assert (row >= 0).all() and (pool.tables[s, pool.nalloc[s]:] == -1).all()
        assert len(set(row.tolist())) == len(row)             # a row never names a block twice
        for b in row:
            counts[b] += 1
    assert (counts == pool.refs).all()
    free = pool.free[:pool.top].tolist()
    assert len(set(free)) == len(free)
    assert set(free) == {b for b in range(pool.n_blocks) if pool.refs[b] == 0}


@pytest.mark.parametrize("seed", range(12))
def test_random_fork_crop_append_isolation(seed):
    rng = np.random.default_rng(seed)
    B, n_seqs, nb, mb = int(rng.choice([1, 4, 16])), 4, 64, 16
    pool = PoolModel(nb, n_seqs, mb, B, n_layers=2, n_kv_heads=1, head_dim=1)
    shadow = [[] for _ in range(n_seqs)]        # logical content: one value per token per layer
    stamp = 0
    for _ in range(60):
        op = rng.integers(0, 3)
        s = int(rng.integers(0, n_seqs))
        if op == 0:                        # append S_i tokens to 1-3 sequences in one call, both layers
            seqs = rng.choice(n_seqs, size=int(rng.integers(1, 4)), replace=False).tolist()
            sizes = [int(rng.integers(1, 2 * B + 3)) for _ in seqs]
            if any(int(pool.lens[q]) + S > mb * B for q, S in zip(seqs, sizes)):
                continue
            before = pool.state()
            rc = pool.reserve(seqs, sizes)
            if rc != OK:
                assert pool.state()["top"] == before["top"]
                continue
            for q, S in zip(seqs, sizes):
                vals = np.arange(stamp, stamp + S, dtype=np.float64)
                stamp += S
                for layer in range(2):
                    kv = (vals + 1000 * layer)[:, None, None]
                    pool.write(layer, q, int(pool.lens[q]), kv, -kv)
                shadow[q] += vals.tolist()
            pool.commit(seqs, sizes)
        elif op == 1:                                             # crop
            L = int(rng.integers(0, int(pool.lens[s]) + 1))
            assert pool.crop([s], [L]) == OK
            shadow[s] = shadow[s][:L]
        else:                                                     # fork s into an empty sequence
            empty = [d for d in range(n_seqs) if pool.lens[d] == 0 and pool.nalloc[d] == 0 and d != s]
            if not empty:
                continue
            d = int(rng.choice(empty))
            assert pool.fork([s], [d]) == OK
            shadow[d] = list(shadow[s])
        _invariants(pool)
        for q in range(n_seqs):
            n = int(pool.lens[q])
            assert n == len(shadow[q])
            for layer in range(2):
                k, v = pool.gather(layer, q, n)
                assert k[:, 0, 0].tolist() == [x + 1000 * layer for x in shadow[q]]
                assert v[:, 0, 0].tolist() == [-(x + 1000 * layer) for x in shadow[q]]


def test_fork_errors_change_nothing():
    pool = PoolModel(16, 4, 4, 4)
    assert pool.reserve([0], [5]) == OK
    pool.commit([0], [5])
    assert pool.fork([0], [1]) == OK
    before = pool.state()
    for srcs, dsts in [([0], [1]), ([0], [0]), ([0, 2], [3, 3]), ([0, 3], [3, 2]), ([0], [4]), ([0, 2], [3])]:
        assert pool.fork(srcs, dsts) == EINVAL
        after = pool.state()
        assert all((after[k] == before[k]).all() for k in before)


@pytest.mark.parametrize("r", [2, 3, 4])
def test_one_reservation_by_every_sharer(r):
    """r rows name one partial tail block; a reservation of all r in one call
    makes r - 1 private copies and the last row in call order writes in place
    (R5, call order), and it needs exactly r - 1 free blocks for them."""
    B = 4
    for order in ([0] + list(range(1, r)), list(range(r - 1, -1, -1))):
        pool = PoolModel(2 + (r - 1), r, 4, B, n_layers=1, n_kv_heads=1, head_dim=1)
        assert pool.reserve([0], [6]) == OK                   # blocks 0, 1; tail of 2 slots
        pool.write(0, 0, 0, np.arange(6.0)[:, None, None], -np.arange(6.0)[:, None, None])
        pool.commit([0], [6])
        assert pool.fork([0] * (r - 1), list(range(1, r))) == OK
        assert pool.top == r - 1 and pool.refs[1] == r
        assert pool.reserve(order, [1] * r) == OK             # one token each, all into the shared tail
        assert pool.top == 0
        assert pool.tables[order[-1], 1] == 1                 # the last one kept the original
        assert len({int(pool.tables[s, 1]) for s in range(r)}) == r
        for i, s in enumerate(order):
            pool.write(0, s, 6, np.array([[[100.0 + i]]]), np.array([[[-100.0 - i]]]))
        pool.commit(order, [1] * r)
        _invariants(pool)
        for i, s in enumerate(order):
            k, v = pool.gather(0, s, 7)
            assert k[:, 0, 0].tolist() == [0, 1, 2, 3, 4, 5, 100 + i]
    # one block short: all-or-nothing ENOMEM
    pool = PoolModel(2 + (r - 2), r, 4, B)
    assert pool.reserve([0], [6]) == OK
    pool.commit([0], [6])
    assert pool.fork([0] * (r - 1), list(range(1, r))) == OK
    before = pool.state()
    assert pool.reserve(list(range(r)), [1] * r) == oracle.ENOMEM
    after = pool.state()
    assert all((after[k] == before[k]).all() for k in before)
