"""Pins of the decoder-layer oracle (oracle/decoder.py): rotary embedding
against its complex-number form and the relative-position identity, RMSNorm's
scale invariance and unit RMS, SiLU against torch's, and whole-layer
properties (zero output projections keep the residual stream; replaying from
any boundary equals the full run, Theorem 1)."""
import numpy as np
import pytest
import torch

from oracle import bf16_round
from oracle import decoder as DEC


def test_rope_matches_complex_rotation():
    rng = np.random.default_rng(0)
    n, h, d, theta = 7, 3, 64, 10000.0
    x = rng.standard_normal((n, h, d))
    pos = rng.integers(0, 40000, size=n)
    got = DEC.rope(x, pos, theta)
    z = x[..., :d // 2] + 1j * x[..., d // 2:]                  # pair i as one complex number
    freqs = np.exp(-np.log(theta) * np.arange(0, d, 2) / d)
    zr = z * np.exp(1j * pos[:, None, None] * freqs[None, None, :])
    assert np.allclose(got, np.concatenate([zr.real, zr.imag], axis=-1), atol=1e-9)
    assert np.allclose(DEC.rope(x, np.zeros(n, int), theta), x)   # position 0 is the identity


def test_rope_relative_position():
    """<R(m) q, R(n) k> = <R(m - n) q, k>: attention sees only offsets."""
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal((1, 1, 128)), rng.standard_normal((1, 1, 128))
    for m, n in [(10, 3), (5000, 4999), (32767, 100)]:
        lhs = np.sum(DEC.rope(q, [m], 5e5) * DEC.rope(k, [n], 5e5))
        rhs = np.sum(DEC.rope(q, [m - n], 5e5) * k)
        assert abs(lhs - rhs) < 1e-8 * max(1.0, abs(lhs))


def test_rms_norm():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 256))
    g = np.ones(256)
    y = DEC.rms_norm(x, g, 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0)
    assert np.allclose(DEC.rms_norm(7.5 * x, g, 0.0), y)
    gain = rng.standard_normal(256)
    assert np.allclose(DEC.rms_norm(x, gain, 1e-5), DEC.rms_norm(x, g, 1e-5) * gain)
    assert (DEC.rms_norm(np.zeros((1, 8)), np.ones(8), 1e-6) == 0).all()


def test_rms_norm_eps_sits_inside_the_root():
    """Hand value at eps != 0 (D2): x = [3, 4], g = 1, eps = 0.5 gives
    mean(x^2) + eps = 12.5 + 0.5 = 13, so y = x / sqrt(13) exactly; eps added
    after the root would give x / (sqrt(12.5) + 0.5) instead."""
    y = DEC.rms_norm(np.array([[3.0, 4.0]]), np.ones(2), 0.5)
    assert np.allclose(y, np.array([[3.0, 4.0]]) / np.sqrt(13.0), rtol=0, atol=1e-15)
    assert not np.allclose(y, np.array([[3.0, 4.0]]) / (np.sqrt(12.5) + 0.5))
    # the library routine with the same convention, at a large eps and a gain
    rng = np.random.default_rng(3)
    x, g = rng.standard_normal((4, 64)), rng.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=0.75).numpy()
    assert np.allclose(DEC.rms_norm(x, g, 0.75), ref, rtol=1e-12, atol=1e-14)


def test_silu_matches_torch():
    g = np.linspace(-30, 30, 1001)
    assert np.allclose(DEC.silu(g), torch.nn.functional.silu(torch.from_numpy(g)).numpy(), rtol=1e-12,
                       atol=1e-15)


def _layers(rng, n_layers, dm, hq, hkv, d, dff, zero_out=False):
    b = lambda *shape, s=1.0: bf16_round(rng.standard_normal(shape) * s)
    out = []
    for _ in range(n_layers):
        w = {"wq": b(dm, hq * d, s=dm ** -0.5), "wk": b(dm, hkv * d, s=dm ** -0.5),
             "wv": b(dm, hkv * d, s=dm ** -0.5), "wo": b(hq * d, dm, s=(hq * d) ** -0.5),
             "wg": b(dm, dff, s=dm ** -0.5), "wu": b(dm, dff, s=dm ** -0.5), "wd": b(dff, dm, s=dff ** -0.5),
             "g_attn": b(dm, s=0.1) + 1.0, "g_mlp": b(dm, s=0.1) + 1.0}
        if zero_out:
            w["wo"] = np.zeros_like(w["wo"])
            w["wd"] = np.zeros_like(w["wd"])
        out.append(w)
    return out


def test_zero_output_projections_keep_the_residual():
    rng = np.random.default_rng(3)
    layers = _layers(rng, 2, 64, 4, 2, 16, 96, zero_out=True)
    x = bf16_round(rng.standard_normal((9, 64)))
    y, _ = DEC.decoder_layers(x, layers, 4, 2, 16, 1e-5, 1e4)
    assert np.array_equal(y, x)


@pytest.mark.parametrize("P", [1, 13, 30])
def test_replay_from_a_boundary_equals_the_full_run(P):
    """Theorem 1 on the oracle: the cache of positions 0..P-1 plus a replay of
    P..T-1 gives the full run's states and keys, exactly."""
    rng = np.random.default_rng(4)
    hq, hkv, d = 4, 2, 16
    layers = _layers(rng, 2, 64, hq, hkv, d, 96)
    x = bf16_round(rng.standard_normal((31, 64)))
    full, kv_full = DEC.decoder_layers(x, layers, hq, hkv, d, 1e-5, 1e4)
    pre, kv_pre = DEC.decoder_layers(x[:P], layers, hq, hkv, d, 1e-5, 1e4)
    rest, kv_rest = DEC.decoder_layers(x[P:], layers, hq, hkv, d, 1e-5, 1e4, pos0=P, cache=kv_pre)
    assert np.array_equal(np.concatenate([pre, rest]), full)
    for (k0, v0), (k1, v1), (kf, vf) in zip(kv_pre, kv_rest, kv_full):
        assert np.array_equal(np.concatenate([k0, k1]), kf) and np.array_equal(np.concatenate([v0, v1]), vf)
