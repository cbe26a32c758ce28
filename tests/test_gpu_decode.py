"""Decode steps (one query token per sequence, the re-decode of model-derived
suffix content: Section 3.2 after Lemma 2, Algorithm 1's replay loop) through
the paged cache: reserve + append of the new token, then attention against
the whole cache, with the keys split across many workgroups and merged in a
fixed order.  Against the fp64 oracle at the bf16 tolerance, and bitwise
reproducible (A1)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import assert_close, dev, log, make_pool, storage_f64

pytestmark = pytest.mark.gpu

GEOM = W.AttnGeometry(32, 8, 128)
SCALE = 128 ** -0.5
GEOM7 = W.AttnGeometry(28, 4, 128)


def _blocks(n, B=16):
    return -(-n // B)


def _prefill(pool, ep, seq):
    P = ep.prefix
    q, k, v = (dev(getattr(ep, x)[:P], "bf16") for x in ("q", "k", "v"))
    assert pool.replay(0, [seq], [P], q, k, v, torch.empty_like(q), SCALE) == 0


def _decode(pool, eps, seqs, steps):
    """Run `steps` decode steps over all sequences; returns [steps, n, Hq, d]."""
    outs = []
    for t in range(steps):
        q, k, v = (torch.cat([dev(getattr(ep, x)[ep.prefix + t:ep.prefix + t + 1], "bf16") for ep in eps])
                   for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, seqs, [1] * len(seqs), q, k, v, o, SCALE) == 0
        outs.append(o)
    return torch.stack(outs)


def _oracle_step(ep, t):
    pos = ep.prefix + t
    return oracle.attention(storage_f64(ep.q[pos:pos + 1], "bf16"), storage_f64(ep.k[:pos + 1], "bf16"),
                            storage_f64(ep.v[:pos + 1], "bf16"), pos, SCALE)


@pytest.mark.parametrize("prefixes", [(8189,), (1000, 4099, 77), (5, 16, 2049, 300, 64, 8191, 1, 700)])
def test_decode_steps_match_oracle(prefixes):
    log(f"decode prefixes={prefixes}")
    steps = 4
    rng = np.random.default_rng(sum(prefixes))
    eps = [W.draw_episode(rng, GEOM, "bf16", P, steps, P + steps) for P in prefixes]
    n = len(eps)
    nb = sum(_blocks(P + steps) + 1 for P in prefixes) + 4
    bps = _blocks(max(prefixes) + steps) + 1
    split = make_pool(GEOM, "bf16", nb, n, bps, split_q=n, max_splits=64)
    plain = make_pool(GEOM, "bf16", nb, n, bps)
    outs = []
    for pool in (split, plain):
        for s, ep in enumerate(eps):
            _prefill(pool, ep, s)
        outs.append(_decode(pool, eps, list(range(n)), steps))
        for s, ep in enumerate(eps):
            assert pool.seq_len(s) == ep.prefix + steps
    for t in range(steps):
        for s, ep in enumerate(eps):
            ref = _oracle_step(ep, t)
            for name, o in zip(("split", "plain"), outs):
                assert_close(o[t, s:s + 1].float().cpu().numpy(), ref, "bf16", f"{name} step {t} seq {s}")
    assert not torch.equal(outs[0], outs[1])       # the split path was taken


def test_decode_group7():
    """Decode at the Qwen2.5-7B geometry (28 / 4 heads, G = 7)."""
    rng = np.random.default_rng(70)
    prefixes, steps = (2000, 45), 3
    eps = [W.draw_episode(rng, GEOM7, "bf16", P, steps, P + steps) for P in prefixes]
    nb = sum(_blocks(P + steps) + 1 for P in prefixes) + 4
    pool = make_pool(GEOM7, "bf16", nb, 2, _blocks(2003) + 1, split_q=2, max_splits=64)
    for s, ep in enumerate(eps):
        _prefill(pool, ep, s)
    out = _decode(pool, eps, [0, 1], steps)
    for t in range(steps):
        for s, ep in enumerate(eps):
            assert_close(out[t, s:s + 1].float().cpu().numpy(), _oracle_step(ep, t), "bf16", f"G7 {t} {s}")


def test_decode_is_bitwise_reproducible():
    rng = np.random.default_rng(5)
    eps = [W.draw_episode(rng, GEOM, "bf16", P, 2, P + 2) for P in (3001, 129)]
    nb = sum(_blocks(ep.prefix + 2) + 1 for ep in eps) + 4
    pool = make_pool(GEOM, "bf16", nb, 2, _blocks(3003) + 1, split_q=2, max_splits=64)
    for s, ep in enumerate(eps):
        _prefill(pool, ep, s)
    first = _decode(pool, eps, [0, 1], 2)
    assert pool.crop([0, 1], [ep.prefix for ep in eps]) == 0
    again = _decode(pool, eps, [0, 1], 2)
    assert torch.equal(first, again)


DEC_CASES = [
    # geometry, block size, prefixes, query tokens per sequence (<= 32 / G: the decode kernel)
    (W.AttnGeometry(32, 8, 128), 16, (0, 5, 100, 1000, 3001), (1, 8, 3, 8, 5)),
    (W.AttnGeometry(28, 4, 128), 32, (31, 777, 2047), (4, 1, 3)),
    (W.AttnGeometry(16, 4, 64), 64, (64, 500, 4000), (7, 2, 8)),
    (W.AttnGeometry(8, 8, 64), 16, (17, 1300), (32, 29)),
]


@pytest.mark.parametrize("case", range(len(DEC_CASES)))
def test_decode_kernel_multi_token_over_poisoned_tails(case):
    """Several query tokens per sequence (causal among themselves) after a crop
    that NaN-fills the released slots: with a workspace the call runs the decode
    kernel (one wave per sequence, KV head and split), without one the prefill
    kernel; both match the oracle, so no stale slot reaches the result."""
    geom, B, prefixes, q_lens = DEC_CASES[case]
    log(f"decode kernel case {case}: {geom} B={B} prefixes={prefixes} q_lens={q_lens}")
    rng = np.random.default_rng(300 + case)
    eps = [W.draw_episode(rng, geom, "bf16", P, S, P + S + 37) for P, S in zip(prefixes, q_lens)]
    n = len(eps)
    nb = sum(-(-ep.t_contaminated // B) + 2 for ep in eps)
    bps = max(-(-ep.t_contaminated // B) for ep in eps) + 1
    scale = geom.head_dim ** -0.5
    seqs = list(range(n))
    cat = lambda f: torch.cat([dev(f(ep), "bf16") for ep in eps])
    outs = []
    for split_q in (sum(q_lens), 0):
        pool = make_pool(geom, "bf16", nb, n, bps, block_size=B, split_q=split_q, max_splits=64)
        cq, ck, cv = (cat(lambda ep, x=x: ep.contaminated(x)) for x in ("q", "k", "v"))
        assert pool.replay(0, seqs, [ep.t_contaminated for ep in eps], cq, ck, cv, torch.empty_like(cq), scale) == 0
        assert pool.crop(seqs, [ep.prefix for ep in eps], poison=True) == 0
        q, k, v = (cat(lambda ep, x=x: getattr(ep, x)[ep.prefix:]) for x in ("q", "k", "v"))
        o = torch.empty_like(q)
        assert pool.replay(0, seqs, list(q_lens), q, k, v, o, scale) == 0
        outs.append(o.float().cpu().numpy())
    off = 0
    for i, ep in enumerate(eps):
        ref = oracle.attention(storage_f64(ep.q[ep.prefix:], "bf16"), storage_f64(ep.k, "bf16"),
                               storage_f64(ep.v, "bf16"), ep.prefix, scale)
        for name, o in zip(("decode kernel", "prefill kernel"), outs):
            got = o[off:off + ep.suffix]
            assert np.isfinite(got).all(), f"{name} seq {i}"
            assert_close(got, ref, "bf16", f"{name} seq {i}")
        off += ep.suffix
