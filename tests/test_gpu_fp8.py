"""FP8 E4M3 KV cache (readings F1, F2): the append stores the E4M3 code of
x / scale per layer, bit for bit as the oracle rounds it (saturation, ties,
subnormals, per-layer scales, copy-on-write copies of codes); attention over
the widened codes times the scales matches the oracle run on the same read-back
values at the bf16 tolerance, through the crop + replay of Algorithm 1 and in
decode steps with split keys; selective replay equals the full reset bitwise."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import assert_close, dev, log, storage_f64

pytestmark = pytest.mark.gpu


def _pool(geom, n_layers, n_blocks, max_seqs, max_bps, B=16, split_q=0, max_splits=16):
    from paper_2609_04875_amd import FP8_E4M3, KVPool, workspace_bytes
    ws = workspace_bytes(geom.n_q_heads, geom.head_dim, split_q, max_splits) if split_q else 0
    return KVPool(n_layers, geom.n_q_heads, geom.n_kv_heads, geom.head_dim, n_blocks, max_seqs, max_bps,
                  FP8_E4M3, B, workspace_bytes=ws)


def _opool(geom, n_layers, n_blocks, max_seqs, max_bps, B=16):
    return oracle.PoolModel(n_blocks, max_seqs, max_bps, B, n_layers=n_layers, n_kv_heads=geom.n_kv_heads,
                            head_dim=geom.head_dim, kv_fp8=True)


def _codes_of(values: np.ndarray) -> np.ndarray:
    """Byte codes of exact E4M3 values (the oracle's stored values)."""
    return torch.from_numpy(np.ascontiguousarray(values)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _device_codes(pool, layer, seq, n):
    """Codes of logical tokens 0..n-1 of ``seq`` as [n, Hkv, d] uint8 (K and V)."""
    torch.cuda.synchronize()
    tables = pool.block_tables[seq].long()
    pos = torch.arange(n, device="cuda")
    blk, slot = tables[pos // pool.B], pos % pool.B
    k = pool.k_cache[layer][blk, :, slot, :]
    v = pool.v_cache[layer][blk, :, :, slot]
    return k.cpu().numpy(), v.cpu().numpy()


def _oracle_codes(opool, layer, seq, n):
    idx = [opool.slot(seq, p) for p in range(n)]
    k = np.stack([opool.kdata[layer, b, o] for b, o in idx])
    v = np.stack([opool.vdata[layer, b, o] for b, o in idx])
    return k, v


def _assert_codes_equal(got: np.ndarray, want_vals: np.ndarray, what: str):
    nan = np.isnan(want_vals)
    want = _codes_of(np.where(nan, 0.0, want_vals))
    assert ((got[nan] & 0x7F) == 0x7F).all(), f"{what}: NaN codes"
    bad = np.flatnonzero((got != want) & ~nan)
    assert bad.size == 0, f"{what}: {bad.size} codes differ, first at {bad[0]}: {got.flat[bad[0]]:#x} vs {want.flat[bad[0]]:#x}"


def _bf16(x: np.ndarray) -> torch.Tensor:
    return dev(W.f32_to_bf16_bits(np.asarray(x, np.float32)), "bf16")


def test_append_codes_bit_exact():
    """Two layers with their own scales; values that saturate, round to
    subnormals, hit exact ties, are -0 or NaN; the device codes equal the
    oracle's, and an unaligned second append lands in the partial block."""
    log("fp8 append codes")
    geom = W.AttnGeometry(8, 2, 64)
    rng = np.random.default_rng(80)
    pool = _pool(geom, 2, 24, 2, 8)
    opool = _opool(geom, 2, 24, 2, 8)
    ks, vs = [0.0173, 0.5], [0.031, 3.0]
    pool.set_kv_scales(ks, vs)
    opool.set_kv_scales(ks, vs)
    for step, (n0, n1) in enumerate([(37, 19), (12, 40)]):
        sizes = [n0, n1]
        S = sum(sizes)
        x = rng.standard_normal((2, S, geom.n_kv_heads, geom.head_dim)).astype(np.float32)
        x[0, :4] *= 40.0                                     # saturating outliers
        x[1, 5:7] *= 1e-4                                    # subnormal codes
        x[0, 8, 0, :8] = np.array([448, 464, 465, -1e4, 0.0, -0.0, 2.0 ** -10, 1.0625], np.float32) * ks[0]
        x[1, 9, 1, :3] = [np.nan, -np.inf, np.inf]
        kb = W.f32_to_bf16_bits(x[0])
        vb = W.f32_to_bf16_bits(x[1])
        q = torch.zeros((S, geom.n_q_heads, geom.head_dim), dtype=torch.bfloat16, device="cuda")
        for layer in (0, 1):
            k, v = dev(kb, "bf16"), dev(vb, "bf16")
            o = torch.empty_like(q)
            assert pool.replay(layer, [0, 1], sizes, q, k, v, o, 0.125, commit=layer == 1) == 0
        kf, vf = storage_f64(kb, "bf16"), storage_f64(vb, "bf16")
        assert opool.reserve([0, 1], sizes) == 0
        off = 0
        for s, n in zip((0, 1), sizes):
            for layer in (0, 1):
                opool.write(layer, s, int(opool.lens[s]), kf[off:off + n], vf[off:off + n])
            off += n
        opool.commit([0, 1], sizes)
        for s in (0, 1):
            L = int(opool.lens[s])
            for layer in (0, 1):
                gk, gv = _device_codes(pool, layer, s, L)
                wk, wv = _oracle_codes(opool, layer, s, L)
                _assert_codes_equal(gk, wk, f"step {step} seq {s} layer {layer} K")
                _assert_codes_equal(gv, wv, f"step {step} seq {s} layer {layer} V")


def _episode_run(geom, B, prefixes, suffixes, contaminated, seed, ks, vs, poison=False):
    """Contaminated prefill, crop (unaligned), sanitized replay on the FP8 pool
    and on the oracle's FP8 pool; returns (device outputs, oracle outputs, eps, pool)."""
    rng = np.random.default_rng(seed)
    eps = [W.draw_episode(rng, geom, "bf16", P, S, C) for P, S, C in zip(prefixes, suffixes, contaminated)]
    n = len(eps)
    nb = sum(-(-max(ep.t_contaminated, ep.prefix + ep.suffix) // B) + 1 for ep in eps) + 2
    bps = max(-(-max(ep.t_contaminated, ep.prefix + ep.suffix) // B) for ep in eps) + 1
    pool = _pool(geom, 1, nb, n, bps, B)
    opool = _opool(geom, 1, nb, n, bps, B)
    pool.set_kv_scales([ks], [vs])
    opool.set_kv_scales([ks], [vs])
    scale = geom.head_dim ** -0.5
    seqs = list(range(n))
    cat = lambda f, dt: torch.cat([dev(f(ep), dt) for ep in eps])
    cq = cat(lambda ep: ep.contaminated("q"), "bf16")
    ck = cat(lambda ep: ep.contaminated("k"), "bf16")
    cv = cat(lambda ep: ep.contaminated("v"), "bf16")
    assert pool.replay(0, seqs, [ep.t_contaminated for ep in eps], cq, ck, cv, torch.empty_like(cq), scale) == 0
    assert pool.crop(seqs, [ep.prefix for ep in eps], poison=poison) == 0
    q = cat(lambda ep: ep.q[ep.prefix:], "bf16")
    k = cat(lambda ep: ep.k[ep.prefix:], "bf16")
    v = cat(lambda ep: ep.v[ep.prefix:], "bf16")
    o = torch.empty_like(q)
    assert pool.replay(0, seqs, [ep.suffix for ep in eps], q, k, v, o, scale) == 0
    # oracle: the same three steps on its own pool
    f = lambda arr: storage_f64(arr, "bf16")
    oracle.prefill(opool, 0, seqs, [ep.t_contaminated for ep in eps],
                   np.concatenate([f(ep.contaminated("q")) for ep in eps]),
                   np.concatenate([f(ep.contaminated("k")) for ep in eps]),
                   np.concatenate([f(ep.contaminated("v")) for ep in eps]), scale)
    assert opool.crop(seqs, [ep.prefix for ep in eps]) == 0
    want = oracle.prefill(opool, 0, seqs, [ep.suffix for ep in eps],
                          np.concatenate([f(ep.q[ep.prefix:]) for ep in eps]),
                          np.concatenate([f(ep.k[ep.prefix:]) for ep in eps]),
                          np.concatenate([f(ep.v[ep.prefix:]) for ep in eps]), scale)
    return o, want, eps, pool, opool


CASES = [
    # geometry, block size, prefixes, suffixes, contaminated lengths, K scale, V scale
    (W.AttnGeometry(32, 8, 128), 16, (260, 0, 1000), (301, 77, 129), (600, 50, 1100), 0.011, 0.013),
    (W.AttnGeometry(28, 4, 128), 32, (97, 513), (200, 64), (300, 520), 1.0, 0.25),
    (W.AttnGeometry(16, 4, 64), 64, (33, 130), (250, 7), (40, 200), 0.02, 2.0),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_fp8_replay_matches_oracle(case):
    geom, B, P, S, C, ks, vs = CASES[case]
    log(f"fp8 replay case {case}: {geom} B={B} prefixes={P} suffixes={S}")
    o, want, eps, pool, opool = _episode_run(geom, B, P, S, C, 800 + case, ks, vs, poison=True)
    off = 0
    for i, ep in enumerate(eps):
        got = o[off:off + ep.suffix].float().cpu().numpy()
        assert_close(got, want[i], "bf16", f"seq {i}")
        off += ep.suffix
        L = ep.prefix + ep.suffix
        gk, gv = _device_codes(pool, 0, i, L)
        wk, wv = _oracle_codes(opool, 0, i, L)
        _assert_codes_equal(gk, wk, f"seq {i} K")
        _assert_codes_equal(gv, wv, f"seq {i} V")


def test_fp8_selective_equals_full_reset_bitwise():
    geom, B, P, S, C, ks, vs = CASES[0]
    log("fp8 selective vs full reset")
    o, _, eps, _, _ = _episode_run(geom, B, P, S, C, 900, ks, vs)
    n = len(eps)
    nb = sum(-(-(ep.prefix + ep.suffix) // B) + 1 for ep in eps) + 2
    full = _pool(geom, 1, nb, n, max(-(-(ep.prefix + ep.suffix) // B) for ep in eps) + 1, B)
    full.set_kv_scales([ks], [vs])
    cat = lambda x: torch.cat([dev(getattr(ep, x), "bf16") for ep in eps])
    fq, fk, fv = cat("q"), cat("k"), cat("v")
    fo = torch.empty_like(fq)
    assert full.full_reset(0, list(range(n)), [ep.prefix + ep.suffix for ep in eps], fq, fk, fv, fo,
                           geom.head_dim ** -0.5) == 0
    off_s, off_f = 0, 0
    for ep in eps:
        a = o[off_s:off_s + ep.suffix]
        b = fo[off_f + ep.prefix:off_f + ep.prefix + ep.suffix]
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
        off_s += ep.suffix
        off_f += ep.prefix + ep.suffix


def test_fp8_decode_split_matches_oracle():
    """Decode steps (one token per sequence) with the keys split over many
    workgroups, against the oracle on the FP8 read-back values."""
    geom = W.AttnGeometry(32, 8, 128)
    log("fp8 decode split")
    rng = np.random.default_rng(81)
    prefixes, steps = (4093, 1, 700), 3
    eps = [W.draw_episode(rng, geom, "bf16", P, steps, P + steps) for P in prefixes]
    n, B = len(eps), 16
    nb = sum(-(-(P + steps) // B) + 1 for P in prefixes) + 2
    bps = -(-(max(prefixes) + steps) // B) + 1
    pool = _pool(geom, 1, nb, n, bps, B, split_q=n, max_splits=64)
    opool = _opool(geom, 1, nb, n, bps, B)
    ks, vs = 0.012, 0.0125
    pool.set_kv_scales([ks], [vs])
    opool.set_kv_scales([ks], [vs])
    scale = 128 ** -0.5
    f = lambda arr: storage_f64(arr, "bf16")
    seqs = list(range(n))
    for s, ep in enumerate(eps):
        P = ep.prefix
        q, k, v = (dev(getattr(ep, x)[:P], "bf16") for x in ("q", "k", "v"))
        assert pool.replay(0, [s], [P], q, k, v, torch.empty_like(q), scale) == 0
        oracle.prefill(opool, 0, [s], [P], f(ep.q[:P]), f(ep.k[:P]), f(ep.v[:P]), scale)
    for t in range(steps):
        sl = lambda ep: slice(ep.prefix + t, ep.prefix + t + 1)
        q, k, v = (torch.cat([dev(getattr(ep, x)[sl(ep)], "bf16") for ep in eps]) for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, seqs, [1] * n, q, k, v, o, scale) == 0
        want = oracle.prefill(opool, 0, seqs, [1] * n, np.concatenate([f(ep.q[sl(ep)]) for ep in eps]),
                              np.concatenate([f(ep.k[sl(ep)]) for ep in eps]),
                              np.concatenate([f(ep.v[sl(ep)]) for ep in eps]), scale)
        for s in range(n):
            assert_close(o[s:s + 1].float().cpu().numpy(), want[s], "bf16", f"step {t} seq {s}")


def test_fp8_fork_copies_codes():
    """Copy-on-write on an FP8 pool: a fork, an unaligned crop of the copy and
    an append into the shared partial block copy codes, not values."""
    geom = W.AttnGeometry(8, 2, 64)
    log("fp8 fork")
    rng = np.random.default_rng(82)
    pool = _pool(geom, 2, 20, 3, 8)
    opool = _opool(geom, 2, 20, 3, 8)
    pool.set_kv_scales([0.02, 0.05], [0.03, 0.07])
    opool.set_kv_scales([0.02, 0.05], [0.03, 0.07])
    f = lambda arr: storage_f64(arr, "bf16")
    L0 = 45

    def put(seqs, sizes):
        S = sum(sizes)
        kb = W.f32_to_bf16_bits(rng.standard_normal((S, 2, 64)).astype(np.float32))
        vb = W.f32_to_bf16_bits(rng.standard_normal((S, 2, 64)).astype(np.float32))
        q = torch.zeros((S, 8, 64), dtype=torch.bfloat16, device="cuda")
        assert opool.reserve(seqs, sizes) == 0
        for layer in (0, 1):
            assert pool.replay(layer, seqs, sizes, q, dev(kb, "bf16"), dev(vb, "bf16"), torch.empty_like(q),
                               0.125, commit=layer == 1) == 0
        off = 0
        for s, n in zip(seqs, sizes):
            for layer in (0, 1):
                opool.write(layer, s, int(opool.lens[s]), f(kb[off:off + n]), f(vb[off:off + n]))
            off += n
        opool.commit(seqs, sizes)

    put([0], [L0])
    assert pool.fork([0], [1]) == 0 and opool.fork([0], [1]) == 0
    assert pool.crop([1], [37]) == 0 and opool.crop([1], [37]) == 0
    put([1, 0], [20, 3])
    st = pool.state()
    assert np.array_equal(st["tables"], opool.tables) and np.array_equal(st["refs"], opool.refs)
    for s in (0, 1):
        L = int(opool.lens[s])
        for layer in (0, 1):
            gk, gv = _device_codes(pool, layer, s, L)
            wk, wv = _oracle_codes(opool, layer, s, L)
            _assert_codes_equal(gk, wk, f"seq {s} layer {layer} K")
            _assert_codes_equal(gv, wv, f"seq {s} layer {layer} V")
