"""Pins of the oracle's FP8 E4M3 rounding (reading F1): every code's value is
a fixed point; in range it equals torch's float8_e4m3fn conversion (a library
routine), ties to even included; past 448 it saturates."""
import numpy as np
import pytest
import torch

import oracle


def _codes():
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_every_code_is_a_fixed_point():
    vals = _codes()
    finite = ~np.isnan(vals)
    assert np.array_equal(oracle.e4m3_round(vals[finite]), vals[finite])
    assert finite.sum() == 254 and np.nanmax(vals) == 448.0


def test_matches_torch_in_range():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * s for s in (1e-3, 0.05, 1, 30, 150)])
    x = x[np.abs(x) <= 460].astype(np.float32).astype(np.float64)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = oracle.e4m3_round(x)
    assert np.array_equal(got, want)
    assert np.array_equal(np.signbit(got), np.signbit(want))


def test_midpoints_round_to_even():
    vals = np.unique(_codes()[~np.isnan(_codes())])
    pos = vals[vals >= 0]
    mids = (pos[:-1] + pos[1:]) / 2                    # exactly halfway between neighbours
    want = torch.from_numpy(mids).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(oracle.e4m3_round(mids), want)
    assert np.array_equal(oracle.e4m3_round(-mids), -want)


def test_saturation_and_nan():
    got = oracle.e4m3_round(np.array([464.0, 465.0, 1e6, np.inf, -np.inf, -500.0, np.nan]))
    assert got[:6].tolist() == [448.0, 448.0, 448.0, 448.0, -448.0, -448.0]
    assert np.isnan(got[6])


# --------------------------------------------------------------------------- #
# The FP8 pool (reading F2): stored codes, per-layer scales, read-back values  #
# --------------------------------------------------------------------------- #
def _code_values(rng, shape, lo=-200.0, hi=200.0):
    vals = _codes()
    vals = vals[~np.isnan(vals) & (vals >= lo) & (vals <= hi)]
    return rng.choice(vals, size=shape)


def test_quantize_matches_torch_fp32_quotient():
    """The stored code of x is torch's float8 conversion of the fp32 quotient."""
    rng = np.random.default_rng(5)
    pool = oracle.PoolModel(4, 1, 4, 16, n_layers=1, n_kv_heads=1, head_dim=8, kv_fp8=True)
    x = oracle.bf16_round(rng.standard_normal(5000) * 3.0)
    for scale in (1.0, 0.0173, 0.5, 3.3):
        want = (torch.from_numpy(x).float() / torch.tensor(scale, dtype=torch.float32))
        keep = (want.abs() <= 448).numpy()               # torch does not saturate (F1)
        want = want.to(torch.float8_e4m3fn).to(torch.float64).numpy()
        assert keep.mean() > 0.9
        assert np.array_equal(pool.quantize(x, scale)[keep], want[keep])


@pytest.mark.parametrize("scale", [0.25, 1.0, 8.0])
def test_lossless_inputs_read_back_exactly(scale):
    """K, V that are code values times a power-of-two scale survive the FP8 pool
    bit for bit, so its prefill equals the full-precision pool's."""
    rng = np.random.default_rng(6)
    B, hq, hkv, d, L = 16, 4, 2, 8, 2
    sizes = [37, 20]
    kw = dict(n_layers=L, n_kv_heads=hkv, head_dim=d)
    p8 = oracle.PoolModel(16, 2, 8, B, kv_fp8=True, **kw)
    p8.set_kv_scales([scale] * L, [scale / 2] * L)
    pf = oracle.PoolModel(16, 2, 8, B, **kw)
    S = sum(sizes)
    q = rng.standard_normal((S, hq, d))
    k = _code_values(rng, (S, hkv, d)) * scale
    v = _code_values(rng, (S, hkv, d)) * (scale / 2)
    for layer in range(L):
        o8 = oracle.prefill(p8, layer, [0, 1], sizes, q, k, v, d ** -0.5, commit=False)
        of = oracle.prefill(pf, layer, [0, 1], sizes, q, k, v, d ** -0.5, commit=False)
        for a, b in zip(o8, of):
            assert np.array_equal(a, b)
    p8.commit([0, 1], sizes)
    kk, vv = p8.gather(1, 0, sizes[0])
    assert np.array_equal(kk, k[:sizes[0]]) and np.array_equal(vv, v[:sizes[0]])


def test_read_back_error_bound_and_layer_scales():
    """Read-back error is at most half a step of the 3-bit mantissa (relative
    2^-4) in the normal range, and each layer uses its own scales."""
    rng = np.random.default_rng(7)
    pool = oracle.PoolModel(4, 1, 4, 16, n_layers=2, n_kv_heads=1, head_dim=16, kv_fp8=True)
    pool.set_kv_scales([0.01, 1.5], [0.02, 3.0])
    pool.reserve([0], [16])
    k = oracle.bf16_round(rng.standard_normal((16, 1, 16)))
    v = oracle.bf16_round(rng.standard_normal((16, 1, 16)))
    for layer in (0, 1):
        pool.write(layer, 0, 0, k, v)
    for layer, ks, vs in ((0, 0.01, 0.02), (1, 1.5, 3.0)):
        kk, vv = pool.gather(layer, 0, 16)
        for got, x, s in ((kk, k, ks), (vv, v, vs)):
            s32 = float(np.float32(s))
            normal = np.abs(x) / s32 >= 2.0 ** -6
            err = np.abs(got - x)
            # the fp32 quotient adds at most 2^-24 relative before the FP8 rounding
            assert (err[normal] <= (2.0 ** -4 + 2.0 ** -23) * np.abs(x[normal])).all()
            assert (err[~normal] <= 2.0 ** -10 * s32 * (1 + 2.0 ** -20)).all()
    # layer 0's scale is small enough that some values saturate at 448 * scale
    big = np.full((16, 1, 16), 10.0)
    pool.write(0, 0, 0, big, big)
    kk, vv = pool.gather(0, 0, 16)
    assert np.allclose(kk, 448 * float(np.float32(0.01))) and np.allclose(vv, 448 * float(np.float32(0.02)))
