"""Pins of the sampling oracle (oracle/sampling.py): Philox4x64-10 against
numpy's Philox bit generator (a library routine; numpy steps its counter
before each block, so its draw from counter c - 1 is the block at c), the
uniform map, Gumbel-max frequencies against softmax(l / T), the greedy limit
and its tie rule."""
import numpy as np
import pytest

from oracle import sampling as S

MASK = (1 << 64) - 1


def _numpy_block(counter, key):
    c = sum(int(w) << (64 * i) for i, w in enumerate(counter)) - 1
    prev = [(c >> (64 * i)) & MASK for i in range(4)]
    bg = np.random.Philox(counter=np.array(prev, dtype=np.uint64), key=np.array(key, dtype=np.uint64))
    return tuple(int(x) for x in bg.random_raw(4))


@pytest.mark.parametrize("counter,key", [
    ((1, 0, 0, 0), (0, 0)), ((0, 1, 0, 0), (0, 0)),          # the second borrows across a word
    ((7, 0, 3, 9), (123456789, 0)), ((MASK, MASK, MASK, MASK), (MASK, MASK)),
    ((0x243F6A8885A308D3, 0x13198A2E03707344, 0xA4093822299F31D0, 0x082EFA98EC4E6C89),
     (0x452821E638D01377, 0xBE5466CF34E90C6C))])
def test_philox_matches_numpy(counter, key):
    assert S.philox4x64_10(counter, key) == _numpy_block(counter, key)


def test_philox_random_counters_match_numpy():
    rng = np.random.default_rng(0)
    for _ in range(50):
        c = tuple(int(x) * 2 + 1 for x in rng.integers(0, 2 ** 63, size=4, dtype=np.int64))
        k = tuple(int(x) for x in rng.integers(0, 2 ** 63, size=2, dtype=np.int64))
        assert S.philox4x64_10(c, k) == _numpy_block(c, k)


def test_uniform_map():
    u = S.uniforms(4003, position=17, stream=2, seed=99)
    assert u.shape == (4003,)
    assert (u > 0).all() and (u < 1).all()
    assert (u.astype(np.float32).astype(np.float64) == u).all()      # fp32-exact
    assert abs(u.mean() - 0.5) < 0.02 and abs((u < 0.25).mean() - 0.25) < 0.03
    words = S.philox4x64_10((1000, 17, 2, 0), (99, 0))
    assert u[4000] == ((words[0] >> 41) + 0.5) / 2 ** 23                # block v div 4, word v mod 4
    assert u[4002] == ((words[2] >> 41) + 0.5) / 2 ** 23
    assert not np.array_equal(u, S.uniforms(4003, position=18, stream=2, seed=99))


@pytest.mark.parametrize("T", [0.7, 1.0, 2.5])
def test_gumbel_max_frequencies_follow_softmax(T):
    logits = np.array([[0.5, -1.0, 2.0, 0.0, 1.0]])
    n = 6000
    toks = [int(S.sample(logits, T, seed=7, streams=[3], positions=[p])[0][0]) for p in range(n)]
    freq = np.bincount(toks, minlength=5) / n
    p = np.exp(logits[0] / T)
    p /= p.sum()
    assert np.abs(freq - p).max() < 0.03, (freq, p)


def test_greedy_and_ties():
    logits = np.array([[0.0, 3.0, 3.0, -1.0], [5.0, 5.0, 5.0, 5.0], [-2.0, -1.0, -3.0, -1.5]])
    toks, gaps = S.sample(logits, 0.0, seed=1, streams=[0, 1, 2], positions=[0, 0, 0])
    assert toks.tolist() == [1, 0, 1]
    assert gaps.tolist() == [0.0, 0.0, 0.5]
    # a very low temperature picks the greedy token
    toks_cold, _ = S.sample(np.array([[0.0, 3.0, 2.5, -1.0]]), 1e-4, seed=1, streams=[0], positions=[5])
    assert toks_cold.tolist() == [1]


def test_same_counter_same_token():
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((4, 300))
    a = S.sample(logits, 0.7, 11, [0, 1, 2, 3], [9, 9, 9, 9])[0]
    b = S.sample(logits, 0.7, 11, [0, 1, 2, 3], [9, 9, 9, 9])[0]
    c = S.sample(logits, 0.7, 12, [0, 1, 2, 3], [9, 9, 9, 9])[0]
    assert (a == b).all() and not (a == c).all()
