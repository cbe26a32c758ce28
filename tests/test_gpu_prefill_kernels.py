"""The bf16 prefill kernels for head_dim 128 and GQA groups dividing 32 (the
wide kernel: one wave per SIMD, 64 rows per wave, 16-token blocks; the
software-pipelined kernel: two waves per SIMD) against the four-wave kernel and
the fp64 oracle.  All kernels take every query row through the same sequence
of operations, so their outputs must agree bit for bit; each must also meet
the bf16 tolerance against the oracle.  Cases cover every group size the pipelined kernel takes, block sizes
16 / 32 / 64, crops not aligned to a block with NaN-poisoned tail slots,
suffixes shorter than one query tile, tiles that straddle the diagonal, and
several sequences of different lengths in one call; then the default kernel
on more shapes against the oracle and against the full reset of every
sequence in one call (bitwise)."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import assert_close, contaminated_then_crop, dev, log, make_pool, oracle_suffix

pytestmark = pytest.mark.gpu


def _blocks(n, B):
    return -(-n // B)


def _run(kind, geom, eps, B, scale):
    """Contaminated prefill, poisoned crop, then one replay call over all
    episodes; returns the per-episode outputs."""
    nb = sum(_blocks(e.t_contaminated, B) + _blocks(e.t_sanitized, B) for e in eps) + 4
    mbps = max(_blocks(max(e.t_contaminated, e.t_sanitized), B) for e in eps) + 2
    pool = make_pool(geom, "bf16", nb, len(eps), mbps, block_size=B)
    pool.set_prefill_kernel(kind)
    for i, e in enumerate(eps):
        contaminated_then_crop(pool, e, i, scale, poison=True)
    q, k, v = (torch.cat([dev(getattr(e, x)[e.prefix:], "bf16") for e in eps]) for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    assert pool.replay(0, list(range(len(eps))), [e.suffix for e in eps], q, k, v, o, scale) == 0
    torch.cuda.synchronize()
    out, off = [], 0
    for e in eps:
        out.append(o[off:off + e.suffix])
        off += e.suffix
    return out


CASES = [
    # (Hq, Hkv, B, [(P, S), ...])
    (32, 8, 16, [(300, 77)]),
    (32, 8, 16, [(0, 130)]),
    (32, 8, 16, [(8189, 96)]),          # the 8B crop point, short suffix
    (32, 8, 16, [(64, 64)]),            # aligned prefix, one query tile
    (32, 32, 16, [(100, 200)]),         # G = 1
    (64, 2, 32, [(50, 70)]),            # G = 32
    (16, 8, 64, [(129, 64)]),           # G = 2, B = 64
    (32, 4, 32, [(1021, 3)]),           # G = 8, fewer queries than one 32-row block
    (64, 4, 16, [(700, 45)]),           # G = 16
    (32, 8, 16, [(517, 90), (0, 33), (2000, 257), (63, 1)]),   # ragged batch in one call
    # more query tiles per KV head than one XCD holds at once (the tiles of a
    # head run in several rounds on its XCD)
    (32, 8, 16, [(5, 2122), (0, 4160)]),
]


@pytest.mark.parametrize("hq,hkv,B,ps", CASES)
def test_pipelined_equals_four_wave_and_oracle(hq, hkv, B, ps):
    geom = W.AttnGeometry(hq, hkv, 128)
    log(f"prefill kernels {hq}/{hkv} B={B} episodes {ps}")
    rng = np.random.default_rng(hq * 7919 + B + sum(p for p, _ in ps))
    eps = [W.draw_episode(rng, geom, "bf16", P, S, P + S + 3) for P, S in ps]
    scale = 128 ** -0.5
    auto = _run("auto", geom, eps, B, scale)          # the wide kernel where B = 16
    pipe = _run("pipelined", geom, eps, B, scale)
    four = _run("four_wave", geom, eps, B, scale)
    for e, a, p, f in zip(eps, auto, pipe, four):
        assert torch.equal(p, f), f"pipelined and four-wave kernels differ (P={e.prefix}, S={e.suffix})"
        assert torch.equal(a, f), f"default and four-wave kernels differ (P={e.prefix}, S={e.suffix})"
        assert_close(a.float().cpu().numpy(), oracle_suffix(e, scale), "bf16", f"P={e.prefix} S={e.suffix}")


# the default kernel on more shapes: the 8B replay at full size, one partial
# query tile, tiles that straddle the diagonal, every group size dividing 16
DEFAULT_CASES = [
    (32, 8, 16, [(8189, 2048)]),         # the 8B replay at full size
    (32, 8, 16, [(300, 31)]),            # one partial query tile
    (32, 8, 16, [(0, 64)]),              # one tile, prefix 0
    (32, 8, 16, [(77, 96)]),             # a tile and a partial one
    (32, 8, 32, [(1000, 130)]),          # B = 32
    (16, 16, 64, [(129, 300)]),          # G = 1, B = 64
    (16, 8, 16, [(50, 150)]),            # G = 2
    (64, 8, 16, [(700, 45)]),            # G = 8
    (64, 4, 16, [(65, 37)]),             # G = 16
    (32, 8, 16, [(517, 90), (0, 33), (2000, 257), (63, 1), (4000, 700)]),   # ragged batch
]


@pytest.mark.parametrize("hq,hkv,B,ps", DEFAULT_CASES)
def test_default_kernel_matches_oracle_and_full_reset(hq, hkv, B, ps):
    geom = W.AttnGeometry(hq, hkv, 128)
    log(f"default kernel {hq}/{hkv} B={B} episodes {ps}")
    rng = np.random.default_rng(hq * 131 + B + sum(p + 3 * s for p, s in ps))
    eps = [W.draw_episode(rng, geom, "bf16", P, S, P + S + 3) for P, S in ps]
    scale = 128 ** -0.5
    outs = _run("auto", geom, eps, B, scale)
    for e, o in zip(eps, outs):
        if e.suffix * hq <= 65536:
            ref, rows = oracle_suffix(e, scale), None
            got = o.float().cpu().numpy()
        else:                                # the full-size case: every 7th row
            rows = np.arange(0, e.suffix * hq, 7)
            ref = oracle_suffix(e, scale, rows=rows)
            got = o.reshape(-1, 128)[torch.from_numpy(rows).cuda()].float().cpu().numpy()
        assert_close(got, ref, "bf16", f"P={e.prefix} S={e.suffix}")
    # Theorem 1, bitwise: the full reset of each sanitized trajectory in one call
    nb = sum(_blocks(e.t_sanitized, B) for e in eps) + 4
    mbps = max(_blocks(e.t_sanitized, B) for e in eps) + 2
    pool = make_pool(geom, "bf16", nb, len(eps), mbps, block_size=B)
    fq, fk, fv = (torch.cat([dev(getattr(e, x), "bf16") for e in eps]) for x in ("q", "k", "v"))
    fo = torch.empty_like(fq)
    assert pool.full_reset(0, list(range(len(eps))), [e.t_sanitized for e in eps], fq, fk, fv, fo,
                           scale) == 0
    torch.cuda.synchronize()
    off = 0
    for e, o in zip(eps, outs):
        assert torch.equal(fo[off + e.prefix:off + e.t_sanitized], o), f"P={e.prefix} S={e.suffix}"
        off += e.t_sanitized


def test_pipelined_full_reset_equals_replay_at_8b_crop():
    """Theorem 1 on the pipelined kernel at the unaligned 8B crop (P = 8189),
    with a suffix spanning several query tiles."""
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(8189)
    P, S = 8189, 640
    ep = W.draw_episode(rng, geom, "bf16", P, S, P + S + 3)
    scale = 128 ** -0.5
    B = 16
    pool = make_pool(geom, "bf16", 2 * _blocks(P + S + 3, B) + 4, 2, _blocks(P + S + 3, B) + 2)
    contaminated_then_crop(pool, ep, 0, scale, poison=True)
    q, k, v = (dev(getattr(ep, x)[P:], "bf16") for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    assert pool.replay(0, [0], [S], q, k, v, o, scale) == 0
    fq, fk, fv = (dev(getattr(ep, x), "bf16") for x in ("q", "k", "v"))
    fo = torch.empty_like(fq)
    assert pool.full_reset(0, [1], [P + S], fq, fk, fv, fo, scale) == 0
    torch.cuda.synchronize()
    assert torch.equal(fo[P:], o)
    rows = np.arange(0, S * 32, 37 * 32 + 5)         # flat (token, head) rows
    ref = oracle_suffix(ep, scale, rows=rows)
    got = o.reshape(S * 32, 128)[torch.from_numpy(rows).cuda()]
    assert_close(got.float().cpu().numpy(), ref, "bf16", "8B crop, sampled rows")


@pytest.mark.parametrize("P,S", [(130700, 100), (130900, 100)])
def test_longest_sequences_for_the_lds_block_table(P, S):
    """A sequence at the wide kernel's limit (130816 keys: a workgroup's copy
    of the block table fills its LDS share) and one just past it (the host
    then runs the pipelined kernel): the default kernel bitwise against the
    four-wave one, and sampled rows against the oracle."""
    geom = W.AttnGeometry(32, 8, 128)
    log(f"longest sequences: P={P} S={S}")
    rng = np.random.default_rng(P)
    eps = [W.draw_episode(rng, geom, "bf16", P, S, P + S + 3)]
    scale = 128 ** -0.5
    auto = _run("auto", geom, eps, 16, scale)[0]
    four = _run("four_wave", geom, eps, 16, scale)[0]
    assert torch.equal(auto, four), f"default and four-wave kernels differ (P={P}, S={S})"
    rows = np.arange(0, S * geom.n_q_heads, 97)
    ref = oracle_suffix(eps[0], scale, rows=rows)
    got = auto.reshape(-1, 128)[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    assert_close(got, ref, "bf16", f"P={P} S={S}")
