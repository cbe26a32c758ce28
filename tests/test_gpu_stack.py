"""Stacked-layer transition F (a reading: the paper defines no layer) on the
GPU: the MFMA GEMM against fp64, and crop + replay of a small stack against
the oracle's stacked layers and against the GPU full reset (Theorem 1,
bitwise: every step is row-independent with a fixed accumulation order)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import assert_close, log

pytestmark = pytest.mark.gpu


def _bf16_dev(a: np.ndarray) -> torch.Tensor:
    bits = W.f32_to_bf16_bits(np.ascontiguousarray(a, np.float32))
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def _f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("m,n,k,res", [(1, 8, 8, False), (37, 136, 72, True), (128, 128, 64, False),
                                       (300, 1024, 520, True), (257, 264, 1024, False),
                                       (1000, 1024, 8192, True), (4100, 4104, 200, True),
                                       # products with at least 256 tiles of 256 x 256 and K a
                                       # multiple of 64 (one wave per SIMD, global->LDS tiles):
                                       # ragged edges with a residual, an odd number of K steps,
                                       # and a single K step
                                       (4100, 4104, 192, True), (4097, 4096, 64, False)])
def test_gemm_matches_fp64(m, n, k, res):
    from paper_2609_04875_amd import gemm_bf16
    rng = np.random.default_rng(m * 7 + n)
    x = rng.standard_normal((m, k)).astype(np.float32)
    w = (rng.standard_normal((n, k)) / np.sqrt(k)).astype(np.float32)     # [n][k]
    r = rng.standard_normal((m, n)).astype(np.float32) if res else None
    xd, wd = _bf16_dev(x), _bf16_dev(w)
    rd = _bf16_dev(r) if res else None
    y = gemm_bf16(xd, wd, r=rd)
    ref = _f64(xd) @ _f64(wd).T + (_f64(rd) if res else 0.0)
    want = oracle.bf16_round(ref)
    got = _f64(y)
    # One bf16 rounding of an fp32 sum vs of the exact sum: one bf16 ulp (taken
    # at the larger magnitude: the two may straddle a power of 2) plus the fp32
    # accumulation error, which is absolute in the size of the terms (it
    # dominates where the sum cancels to near zero).
    ulp = np.maximum(np.abs(want), np.abs(got)) * 2.0 ** -7
    terms = np.abs(_f64(xd)) @ np.abs(_f64(wd)).T + (np.abs(_f64(rd)) if res else 0.0)
    bound = ulp + 2.0 ** -20 * terms
    assert np.all(np.abs(got - want) <= bound), np.abs(got - want).max()
    assert np.mean(got == want) > 0.95


def test_gemm_rows_are_independent_and_deterministic():
    from paper_2609_04875_amd import gemm_bf16
    rng = np.random.default_rng(3)
    x = _bf16_dev(rng.standard_normal((333, 512)))
    w = _bf16_dev(rng.standard_normal((256, 512)) / 20)
    full = gemm_bf16(x, w)
    assert torch.equal(full, gemm_bf16(x, w))
    part = gemm_bf16(x[101:230].contiguous(), w)
    assert torch.equal(part, full[101:230])


def test_gemm_tile_shapes_agree_bitwise():
    """A product large enough for the one-wave-per-SIMD kernel (16 x 16 tiles
    of 256 x 256) and a slice of its rows, which runs the register-staged
    kernel's 128 x 128 tiles: same bits per row."""
    from paper_2609_04875_amd import gemm_bf16
    rng = np.random.default_rng(5)
    x = _bf16_dev(rng.standard_normal((4096, 1024)))
    w = _bf16_dev(rng.standard_normal((4096, 1024)) / 32)
    full = gemm_bf16(x, w)
    part = gemm_bf16(x[1000:1300].contiguous(), w)
    assert torch.equal(part, full[1000:1300])


@pytest.mark.parametrize("rows", [(101, 201), (7, 70), (0, 1), (40, 168)])
def test_gemm_narrow_tiles_agree_bitwise(rows):
    """Few rows (64 x 32 or 128 x 32 tiles) against the same rows inside a
    larger product (128 x 128 tiles): same bits; K not a multiple of 64."""
    from paper_2609_04875_amd import gemm_bf16
    rng = np.random.default_rng(6)
    x = _bf16_dev(rng.standard_normal((4096, 1000)))       # 32 x 9 tiles of 128 x 128
    w = _bf16_dev(rng.standard_normal((1048, 1000)) / 32)
    r = _bf16_dev(rng.standard_normal((4096, 1048)))
    full = gemm_bf16(x, w, r=r)
    a, b = rows
    part = gemm_bf16(x[a:b].contiguous(), w, r=r[a:b].contiguous())
    assert torch.equal(part, full[a:b])


@pytest.mark.parametrize("m,n,k", [(64, 128, 256), (4096, 4096, 128)])   # both kernels
def test_gemm_residual_may_alias_output(m, n, k):
    from paper_2609_04875_amd import gemm_bf16
    rng = np.random.default_rng(4)
    x = _bf16_dev(rng.standard_normal((m, k)))
    w = _bf16_dev(rng.standard_normal((n, k)) / 16)
    r = _bf16_dev(rng.standard_normal((m, n)))
    want = gemm_bf16(x, w, r=r)
    gemm_bf16(x, w, r=r, out=r)
    assert torch.equal(r, want)


def _small_stack(T=300, dm=1024, layers=3, seed=9):
    geom = W.AttnGeometry(8, 1, 128)
    w = W.Workload("small_stack", geom, "bf16", seed=seed, n_layers=layers, d_model=dm, t_total=T)
    x0, xc, ws = W.stack_inputs(w)
    return geom, w, x0, xc, ws


def test_stack_replay_matches_oracle_and_full_reset():
    from paper_2609_04875_amd import StackedReplay
    geom, w, x0, xc, ws = _small_stack()
    T, P = 300, 203
    log(f"small stack T={T} P={P}")
    f32 = lambda b: W.bf16_bits_to_f32(b)
    wdev = [tuple(_bf16_dev(f32(m).T) for m in layer) for layer in ws]   # [out][in] layout
    stack = StackedReplay(wdev, geom.n_q_heads, geom.n_kv_heads, geom.head_dim,
                          n_blocks=2 * (-(-T // 16)) + 8, max_seqs=2, max_blocks_per_seq=32)
    scale = 128 ** -0.5
    xs = _bf16_dev(f32(x0))
    xcont = _bf16_dev(np.concatenate([f32(x0)[:P], f32(xc)[P:]]))
    stack.replay(0, xcont, scale)                       # contaminated run into the cache
    assert stack.crop([0], [P]) == 0                    # restore to tau - 1
    out = stack.replay(0, xs[P:].contiguous(), scale)   # sanitized suffix
    assert stack.pool.seq_len(0) == T
    full = stack.full_reset(1, xs, scale)
    assert torch.equal(full[P:], out)                   # Theorem 1, bitwise
    # oracle: the sanitized trajectory through the stacked layers
    layers64 = [tuple(f32(m).astype(np.float64) for m in layer) for layer in ws]
    ref, _ = oracle.stacked_layers(f32(x0).astype(np.float64), layers64, geom.n_q_heads,
                                   geom.n_kv_heads, geom.head_dim, scale)
    # The layer state x is a bf16 residual stream (magnitudes past 8 after three
    # layers).  GPU and fp64 differ by fp32 accumulation, bf16 P in attention
    # and storage-rounding flips that later layers carry on; where x + O Wo
    # cancels to ~0 the elementwise relative error is meaningless.  Bound: two
    # bf16 ulps at the largest magnitude, and L1-relative error 1e-2.
    got, want = _f64(out), ref[P:]
    d = np.abs(got - want)
    assert d.max() <= 2.0 ** -6 * np.abs(want).max(), (d.max(), np.abs(want).max())
    assert d.sum() / np.abs(want).sum() <= 1e-2


def test_stack_at_the_70b_geometry_matches_oracle():
    """The stacked workload's own geometry (64 query / 8 KV heads, d 128,
    d_model 8192) at a reduced T = 2048 and 2 layers: crop to 25 % and 95 % of
    T (the latter unaligned) and replay, against the oracle's stack over the
    whole sanitized trajectory; each layer's attention output also within the
    bf16 attention tolerance (max |d| <= 2e-2, sum|d| / sum|ref| <= 1e-2), and
    the replays bitwise equal to the GPU full reset (Theorem 1)."""
    from paper_2609_04875_amd import StackedReplay
    base = W.workload("stack70b_8layer_t16384_bf16")
    T, L = 2048, 2
    geom, dm = base.geometry, base.d_model
    w = W.Workload("stack70b_2layer_t2048", geom, "bf16", seed=base.seed, n_layers=L, d_model=dm, t_total=T)
    log(f"70B-geometry stack: T={T}, {L} layers, d_model {dm}")
    x0, xc, ws = W.stack_inputs(w)
    f32 = lambda b: W.bf16_bits_to_f32(b)
    dev = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).cuda()
    wdev = [tuple(dev(np.ascontiguousarray(m.T)) for m in layer) for layer in ws]   # [out][in]
    nb = -(-T // 16)
    stack = StackedReplay(wdev, geom.n_q_heads, geom.n_kv_heads, geom.head_dim,
                          n_blocks=3 * nb + 8, max_seqs=3, max_blocks_per_seq=nb + 2)
    scale = base.scale
    xs = dev(x0)
    full_att = []
    full = stack.full_reset(2, xs, scale, record=full_att)
    crops = [int(T * 0.25), int(np.floor(T * 0.95))]           # 512 and 1945 (9 valid in the tail block)
    outs = {}
    for seq, P in enumerate(crops):
        xcont = dev(np.concatenate([x0[:P], xc[P:]]))
        stack.replay(seq, xcont, scale)                           # contaminated run into the cache
        assert stack.crop([seq], [P]) == 0
        att = []
        out = stack.replay(seq, xs[P:].contiguous(), scale, record=att)
        assert stack.pool.seq_len(seq) == T
        assert torch.equal(full[P:], out)                         # Theorem 1, bitwise
        for a, fa in zip(att, full_att):
            assert torch.equal(fa[P:], a)
        outs[P] = (out, att)
    log("oracle: 2 layers over 2048 tokens in fp64")
    layers64 = [tuple(f32(m).astype(np.float64) for m in layer) for layer in ws]
    ref_att = []
    ref, _ = oracle.stacked_layers(f32(x0).astype(np.float64), layers64, geom.n_q_heads,
                                   geom.n_kv_heads, geom.head_dim, scale, record=ref_att)
    for P, (out, att) in outs.items():
        for li, (a, ra) in enumerate(zip(att, ref_att)):
            assert_close(_f64(a), ra[P:], "bf16", f"P={P}: attention output of layer {li}")
        got, want = _f64(out), ref[P:]
        d = np.abs(got - want)
        log(f"P={P}: final state max|d| {d.max():.3e} (|ref| max {np.abs(want).max():.2f}), "
            f"L1-rel {d.sum() / np.abs(want).sum():.3e}")
        assert d.max() <= 2.0 ** -6 * np.abs(want).max()
        assert d.sum() / np.abs(want).sum() <= 1e-2
