"""Full decoder layers on the GPU against the fp64 oracle (oracle/decoder.py):
the elementwise kernels (RMSNorm, rotary embedding at absolute positions,
SwiGLU gate) to one bf16 rounding, and replay through two full layers at a
G = 2 and a G = 7 geometry against the oracle and bitwise against the full
reset (Theorem 1)."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import bf16_round
from oracle import decoder as DEC
from gpu_helpers import log

from paper_2609_04875_amd import DecoderReplay, rmsnorm, rope_, silu_mul

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda().to(torch.bfloat16)


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _within_one_rounding(got, want):
    """got is want's fp32 value rounded once to bf16: within one bf16 step of
    the exact value (2^-8 relative), plus a floor for values near 0."""
    d = np.abs(got - want)
    assert (d <= 2.0 ** -8 * np.abs(want) + 1e-6).all(), (d.max(), np.argmax(d))


def test_rmsnorm_matches_oracle():
    rng = np.random.default_rng(0)
    x = bf16_round(rng.standard_normal((37, 4096)) * 3)
    g = bf16_round(1 + 0.1 * rng.standard_normal(4096))
    got = _f64(rmsnorm(_dev(x), _dev(g), 1e-5))
    _within_one_rounding(got, DEC.rms_norm(x, g, 1e-5))


def test_rope_matches_oracle_at_large_positions():
    rng = np.random.default_rng(1)
    x = bf16_round(rng.standard_normal((50, 8, 128)))
    pos = rng.integers(0, 131072, size=50).astype(np.int32)
    t = _dev(x)
    rope_(t, torch.from_numpy(pos).cuda(), 5e5)
    _within_one_rounding(_f64(t), DEC.rope(x, pos, 5e5))


def test_silu_mul_matches_oracle():
    rng = np.random.default_rng(2)
    gu = bf16_round(rng.standard_normal((19, 2 * 1024)) * 4)
    got = _f64(silu_mul(_dev(gu)))
    _within_one_rounding(got, DEC.silu(gu[:, :1024]) * gu[:, 1024:])


def _weights(rng, n_layers, dm, hq, hkv, d, dff):
    b = lambda *shape, s=1.0: bf16_round(rng.standard_normal(shape) * s)
    ws = []
    for _ in range(n_layers):
        ws.append({"wq": b(dm, hq * d, s=dm ** -0.5), "wk": b(dm, hkv * d, s=dm ** -0.5),
                   "wv": b(dm, hkv * d, s=dm ** -0.5), "wo": b(hq * d, dm, s=(hq * d) ** -0.5),
                   "wg": b(dm, dff, s=dm ** -0.5), "wu": b(dm, dff, s=dm ** -0.5),
                   "wd": b(dff, dm, s=dff ** -0.5),
                   "g_attn": bf16_round(1 + 0.1 * rng.standard_normal(dm)),
                   "g_mlp": bf16_round(1 + 0.1 * rng.standard_normal(dm))})
    return ws


def _dev_weights(ws):
    return [{"wq": _dev(w["wq"].T), "wk": _dev(w["wk"].T), "wv": _dev(w["wv"].T), "wo": _dev(w["wo"].T),
             "w_gate_up": _dev(np.concatenate([w["wg"].T, w["wu"].T])), "w_down": _dev(w["wd"].T),
             "g_attn": _dev(w["g_attn"]), "g_mlp": _dev(w["g_mlp"])} for w in ws]


@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 64), (7, 1, 64)])
def test_decoder_replay_matches_oracle_and_full_reset(hq, hkv, d):
    log(f"decoder layers {hq}/{hkv}/{d}")
    rng = np.random.default_rng(hq)
    dm, dff, T, P, Tc = hq * d, 384, 300, 203, 330
    eps, theta = 1e-5, 5e5
    ws = _weights(rng, 2, dm, hq, hkv, d, dff)
    x = bf16_round(rng.standard_normal((T, dm)))
    xc = np.concatenate([x[:P], bf16_round(rng.standard_normal((Tc - P, dm)))])   # contaminated run
    dec = DecoderReplay(_dev_weights(ws), hq, hkv, d, eps, theta, n_blocks=2 * (-(-Tc // 16)) + 8,
                        max_seqs=2, max_blocks_per_seq=32)
    dec.replay(0, _dev(xc))
    assert dec.crop([0], [P]) == 0
    out = dec.replay(0, _dev(x[P:]))
    full = dec.full_reset(1, _dev(x))
    torch.cuda.synchronize()
    assert torch.equal(full[P:], out)                                 # Theorem 1, bitwise
    assert dec.pool.seq_len(0) == T and dec.pool.seq_len(1) == T
    ref, _ = DEC.decoder_layers(x, ws, hq, hkv, d, eps, theta)
    got, want = _f64(out), ref[P:]
    diff = np.abs(got - want)
    # the residual stream after two layers: two bf16 steps at the largest
    # magnitude, L1-relative 1e-2 (as for the stacked layers)
    assert diff.max() <= 2.0 ** -6 * np.abs(want).max(), (diff.max(), np.abs(want).max())
    assert diff.sum() / np.abs(want).sum() <= 1e-2


def test_captured_restore_replay_matches_eager():
    """Restore + replay through two layers recorded as one HIP graph: three
    replays, each from the restored contaminated state with eager library work
    in between, give the eager replay's bits every time."""
    log("decoder restore + replay as a HIP graph")
    hq, hkv, d = 4, 2, 64
    rng = np.random.default_rng(99)
    dm, dff, T, P, Tc = hq * d, 384, 300, 203, 330
    eps, theta = 1e-5, 5e5
    ws = _weights(rng, 2, dm, hq, hkv, d, dff)
    x = bf16_round(rng.standard_normal((T, dm)))
    xc = np.concatenate([x[:P], bf16_round(rng.standard_normal((Tc - P, dm)))])
    dec = DecoderReplay(_dev_weights(ws), hq, hkv, d, eps, theta, n_blocks=3 * (-(-Tc // 16)) + 8,
                        max_seqs=2, max_blocks_per_seq=32)
    dec.replay(0, _dev(xc))
    torch.cuda.synchronize()
    saved = dec.pool.save_meta()
    assert dec.crop([0], [P]) == 0
    want = dec.replay(0, _dev(x[P:])).clone()
    torch.cuda.synchronize()
    after = dec.pool.save_meta()

    dec.pool.load_meta(saved)
    cap = dec.capture_restore_replay(0, P, _dev(x[P:]))
    for i in range(3):
        dec.pool.load_meta(saved)
        got = cap.replay()
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"graph replay {i} differs from the eager replay"
        assert all(torch.equal(a, b) for a, b in zip(dec.pool.save_meta(), after)), f"replay {i} tables"
        # eager work between replays: a full reset of another sequence
        dec.pool.refresh()
        full = dec.full_reset(1, _dev(x))
        torch.cuda.synchronize()
        assert torch.equal(full[P:], want)
        assert dec.crop([1], [0]) == 0
        torch.cuda.synchronize()
