"""Pins of the stacked random-init layer F (a reading: the paper defines no layer;
parity against the paper is unpinned).  Pinned by special cases with closed
forms and by Theorem 1 (splicing equivalence) on the stack itself."""
import numpy as np

import oracle


def _layers(rng, L, dm, hq, hkv, d, zero_q=False, zero_o=False):
    out = []
    for _ in range(L):
        wq = np.zeros((dm, hq * d)) if zero_q else oracle.bf16_round(rng.standard_normal((dm, hq * d)) / np.sqrt(dm))
        wk = oracle.bf16_round(rng.standard_normal((dm, hkv * d)) / np.sqrt(dm))
        wv = oracle.bf16_round(rng.standard_normal((dm, hkv * d)) / np.sqrt(dm))
        wo = np.zeros((hq * d, dm)) if zero_o else oracle.bf16_round(rng.standard_normal((hq * d, dm)) / np.sqrt(dm))
        out.append((wq, wk, wv, wo))
    return out


def test_zero_output_projection_keeps_the_residual():
    rng = np.random.default_rng(0)
    x = oracle.bf16_round(rng.standard_normal((12, 32)))
    y, kv = oracle.stacked_layers(x, _layers(rng, 2, 32, 4, 2, 8, zero_o=True), 4, 2, 8, 8 ** -0.5)
    np.testing.assert_array_equal(y, x)
    assert kv[0][0].shape == (12, 2, 8)


def test_zero_query_projection_gives_causal_mean_of_values():
    rng = np.random.default_rng(1)
    dm, hq, hkv, d, n = 32, 4, 2, 8, 10
    x = oracle.bf16_round(rng.standard_normal((n, dm)))
    layers = _layers(rng, 1, dm, hq, hkv, d, zero_q=True)
    wq, wk, wv, wo = layers[0]
    y, _ = oracle.stacked_layers(x, layers, hq, hkv, d, d ** -0.5)
    v = oracle.bf16_round(x @ wv).reshape(n, hkv, d)
    mean = np.cumsum(v, axis=0) / np.arange(1, n + 1)[:, None, None]
    o = oracle.bf16_round(np.repeat(mean, hq // hkv, axis=1).reshape(n, hq * d))
    np.testing.assert_allclose(y, oracle.bf16_round(x + o @ wo), rtol=0, atol=0)


def test_theorem1_on_the_stack():
    # Replay from P with the per-layer cached prefix K/V equals the full run.
    rng = np.random.default_rng(2)
    dm, hq, hkv, d, T, P = 32, 4, 2, 8, 20, 13
    layers = _layers(rng, 3, dm, hq, hkv, d)
    x = oracle.bf16_round(rng.standard_normal((T, dm)))
    full, kv = oracle.stacked_layers(x, layers, hq, hkv, d, d ** -0.5)
    part, _ = oracle.stacked_layers(x[P:], layers, hq, hkv, d, d ** -0.5, pos0=P, cache=kv)
    # row-subset matmuls may round differently inside BLAS; bf16 storage rounding
    # can then flip by one ulp, which the check allows
    np.testing.assert_allclose(part, full[P:], rtol=2 ** -7, atol=1e-6)
    assert np.mean(part == full[P:]) > 0.99
