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
        if op == 0:                                               # append S tokens on both layers
            S = int(rng.integers(1, 2 * B + 3))
            P = int(pool.lens[s])
            if P + S > mb * B:
                continue
            before = pool.state()
            rc = pool.reserve([s], [S])
            if rc != OK:
                assert pool.state()["top"] == before["top"]
                continue
            vals = np.arange(stamp, stamp + S, dtype=np.float64)
            stamp += S
            for layer in range(2):
                kv = (vals + 1000 * layer)[:, None, None]
                pool.write(layer, s, P, kv, -kv)
            pool.commit([s], [S])
            shadow[s] += vals.tolist()
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
