"""Calls with more sequences than one launch carries (64), through the
split-key and decode paths whose partials are merged by a separate combine
launch.  Each launch owns one contiguous run of the packed query rows; every
row of the call is compared with the fp64 oracle, so a combine that touched
another launch's rows would show here.  Same softmax attention as the plain
path (Section 3.2, replay by prefill), so the bf16 / fp32 tolerances apply."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import assert_close, dev, log, make_pool, storage_f64

pytestmark = pytest.mark.gpu


def _blocks(n, B=16):
    return -(-n // B)


CASES = [
    # name, geometry, dtype, sequences, prefix range, query-length range, bf16 kernel choice
    # decode: every query length <= 32 / G, pool with a workspace -> decode
    # kernel with key splits, 64 + 16 sequences in two launches
    ("decode", W.AttnGeometry(4, 1, 64), "bf16", 80, (700, 1400), (1, 8), "auto"),
    # wide bf16 prefill (16-token blocks) with split keys (few tiles per launch), 64 + 6
    ("prefill_wide", W.AttnGeometry(8, 2, 128), "bf16", 70, (300, 900), (1, 60), "auto"),
    # the two-wave pipelined kernel on the same shapes
    ("prefill_pipe", W.AttnGeometry(8, 2, 128), "bf16", 70, (300, 900), (1, 60), "pipelined"),
    # four-wave bf16 kernel (head_dim 64), 64 + 66 + 2 sequences in three launches
    ("prefill_four_wave", W.AttnGeometry(8, 2, 64), "bf16", 130, (100, 500), (1, 40), "auto"),
    # fp32 kernel with split keys, 64 + 2
    ("prefill_f32", W.AttnGeometry(4, 2, 64), "f32", 66, (100, 400), (1, 40), "auto"),
]


@pytest.mark.parametrize("name,geom,dtype,n,p_rng,s_rng,kernel", CASES, ids=[c[0] for c in CASES])
def test_many_sequences_split_and_decode_match_oracle(name, geom, dtype, n, p_rng, s_rng, kernel):
    log(f"many sequences: {name}, {n} sequences")
    rng = np.random.default_rng(len(name) * 100 + n)
    P = rng.integers(p_rng[0], p_rng[1] + 1, size=n).tolist()
    S = rng.integers(s_rng[0], s_rng[1] + 1, size=n).tolist()
    eps = [W.draw_episode(rng, geom, dtype, p, s, p) for p, s in zip(P, S)]
    scale = geom.head_dim ** -0.5
    nb = sum(_blocks(p + s) for p, s in zip(P, S)) + 8
    mbps = max(_blocks(p + s) for p, s in zip(P, S)) + 1
    order = rng.permutation(n).tolist()            # packed in another order than the ids
    outs = []
    for split_q in (sum(S), 0):                    # with and without a workspace
        pool = make_pool(geom, dtype, nb, n, mbps, split_q=split_q, max_splits=32)
        if dtype == "bf16":
            pool.set_prefill_kernel(kernel)
        seqs = list(range(n))
        pq = torch.cat([dev(e.q[:e.prefix], dtype) for e in eps])
        pk = torch.cat([dev(e.k[:e.prefix], dtype) for e in eps])
        pv = torch.cat([dev(e.v[:e.prefix], dtype) for e in eps])
        assert pool.replay(0, seqs, P, pq, pk, pv, torch.empty_like(pq), scale) == 0
        q = torch.cat([dev(eps[i].q[eps[i].prefix:], dtype) for i in order])
        k = torch.cat([dev(eps[i].k[eps[i].prefix:], dtype) for i in order])
        v = torch.cat([dev(eps[i].v[eps[i].prefix:], dtype) for i in order])
        o = torch.full_like(q, float("nan"))
        assert pool.replay(0, order, [S[i] for i in order], q, k, v, o, scale) == 0
        torch.cuda.synchronize()
        outs.append(o)
        got = o.float().cpu().numpy()
        off = 0
        for i in order:
            e = eps[i]
            ref = oracle.attention(storage_f64(e.q[e.prefix:], dtype), storage_f64(e.k, dtype),
                                   storage_f64(e.v, dtype), e.prefix, scale)
            assert_close(got[off:off + e.suffix], ref, dtype, f"{name} split_q={split_q} sequence {i}")
            off += e.suffix
    # the workspace pool really took the split / decode path (else this test
    # would not cover the combine)
    assert not torch.equal(outs[0], outs[1])
