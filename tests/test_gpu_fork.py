"""Copy-on-write fork on the GPU (pgsr_kv_fork; reading R5 of the oracle
pool): device block tables, lengths, free-list stack and block counts equal
the oracle's bit for bit after every random fork / crop / append, and every
sequence's cached K/V (read through the device table) equals the oracle's;
then the paper's use: branches of one contaminated base replay selectively
and fully (Theorem 1, bitwise) while the base stays untouched."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import assert_close, bits, dev, log, logical_kv, make_pool, oracle_suffix

pytestmark = pytest.mark.gpu


def _state_eq(pool, opool, what):
    st, ost = pool.state(), opool.state()
    top = ost["top"]
    assert (st["tables"] == ost["tables"]).all(), what
    assert (st["lens"] == ost["lens"]).all(), what
    assert st["top"] == top, what
    assert (st["free"][:top] == ost["free"][:top]).all(), what
    assert (st["refs"] == ost["refs"]).all(), what


@pytest.mark.parametrize("seed", range(6))
def test_random_fork_crop_append_match_oracle(seed):
    log(f"fork random ops seed={seed}")
    rng = np.random.default_rng(seed)
    geom = W.AttnGeometry(4, 2, 64)
    B, n_seqs, nb, mbps, layers = 16, 4, 48, 12, 2
    pool = make_pool(geom, "f32", nb, n_seqs, mbps, n_layers=layers, block_size=B)
    opool = oracle.PoolModel(nb, n_seqs, mbps, B, n_layers=layers, n_kv_heads=2, head_dim=64)
    for step in range(40):
        op = int(rng.integers(0, 3))
        s = int(rng.integers(0, n_seqs))
        if op == 0:                          # append S_i tokens to 1-3 sequences in one call, both layers
            seqs = rng.choice(n_seqs, size=int(rng.integers(1, 4)), replace=False).tolist()
            sizes = [int(rng.integers(1, 2 * B + 5)) for _ in seqs]
            if any(int(opool.lens[q]) + S > mbps * B for q, S in zip(seqs, sizes)):
                continue
            starts = [int(opool.lens[q]) for q in seqs]
            rc_o = opool.reserve(seqs, sizes)
            T = sum(sizes)
            for layer in range(layers):
                k = rng.standard_normal((T, 2, 64)).astype(np.float32)
                v = rng.standard_normal((T, 2, 64)).astype(np.float32)
                q = rng.standard_normal((T, 4, 64)).astype(np.float32)
                o = torch.empty((T, 4, 64), device="cuda")
                rc = pool.replay(layer, seqs, sizes, dev(q, "f32"), dev(k, "f32"), dev(v, "f32"), o,
                                 0.125, commit=layer == layers - 1)
                assert rc == rc_o, (rc, rc_o)                      # ENOMEM on both sides, or neither
                if rc:
                    break
                off = 0
                for qs, P, S in zip(seqs, starts, sizes):
                    opool.write(layer, qs, P, k[off:off + S].astype(np.float64), v[off:off + S].astype(np.float64))
                    off += S
            if rc_o == 0:
                opool.commit(seqs, sizes)
        elif op == 1:                                          # crop
            L = int(rng.integers(0, int(opool.lens[s]) + 1))
            assert opool.crop([s], [L]) == 0
            assert pool.crop([s], [L]) == 0
        else:                                                  # fork into an empty sequence
            empty = [d for d in range(n_seqs) if opool.lens[d] == 0 and opool.nalloc[d] == 0 and d != s]
            if not empty:
                continue
            d = int(rng.choice(empty))
            assert opool.fork([s], [d]) == 0
            assert pool.fork([s], [d]) == 0
        _state_eq(pool, opool, f"step {step} op {op}")
        for q in range(n_seqs):
            n = int(opool.lens[q])
            for layer in range(layers):
                k, v = logical_kv(pool, layer, q, n)
                ok, ov = opool.gather(layer, q, n)
                assert np.array_equal(k.cpu().numpy().astype(np.float64), ok), (step, q, layer)
                assert np.array_equal(v.cpu().numpy().astype(np.float64), ov), (step, q, layer)


def test_branches_of_one_base():
    """Two forks of a contaminated base: one crops to the unaligned boundary and
    replays the suffix, the other replays everything from 0.  Their suffix
    outputs agree bitwise (Theorem 1), match the oracle, and the base's cache
    is unchanged."""
    geom = W.AttnGeometry(32, 8, 128)
    rng = np.random.default_rng(17)
    P, S, Tc = 1021, 300, 1400
    ep = W.draw_episode(rng, geom, "bf16", P, S, Tc)
    scale = 128 ** -0.5
    nb = -(-Tc // 16) + 2 * (-(-(P + S) // 16)) + 8
    pool = make_pool(geom, "bf16", nb, 3, 128)
    cq, ck, cv = (dev(ep.contaminated(x), "bf16") for x in ("q", "k", "v"))
    assert pool.replay(0, [0], [Tc], cq, ck, cv, torch.empty_like(cq), scale) == 0
    base_k, base_v = (t.clone() for t in logical_kv(pool, 0, 0, Tc))
    assert pool.fork([0, 0], [1, 2]) == 0
    assert pool.state()["refs"][pool.state()["tables"][0][:-(-Tc // 16)]].tolist() == [3] * (-(-Tc // 16))
    assert pool.crop([1], [P]) == 0
    q, k, v = (dev(getattr(ep, x)[P:], "bf16") for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    assert pool.replay(0, [1], [S], q, k, v, o, scale) == 0           # copy-on-write of block 63
    fq, fk, fv = (dev(getattr(ep, x), "bf16") for x in ("q", "k", "v"))
    fo = torch.empty_like(fq)
    assert pool.full_reset(0, [2], [P + S], fq, fk, fv, fo, scale) == 0
    torch.cuda.synchronize()
    assert torch.equal(fo[P:], o)
    assert_close(o.float().cpu().numpy(), oracle_suffix(ep, scale), "bf16", "fork replay")
    k0, v0 = logical_kv(pool, 0, 0, Tc)
    assert torch.equal(k0, base_k) and torch.equal(v0, base_v)        # the base is untouched
    assert pool.seq_len(0) == Tc and pool.seq_len(1) == P + S and pool.seq_len(2) == P + S


def test_fork_errors_change_nothing():
    geom = W.AttnGeometry(4, 2, 64)
    pool = make_pool(geom, "f32", 16, 4, 4)
    x = torch.zeros((20, 2, 64), device="cuda")
    assert pool.replay(0, [0], [20], torch.zeros((20, 4, 64), device="cuda"), x, x,
                       torch.empty((20, 4, 64), device="cuda"), 0.125) == 0
    assert pool.fork([0], [1]) == 0
    before = pool.state()
    for srcs, dsts in [([0], [1]), ([0], [0]), ([2, 0], [3, 3]), ([0, 3], [3, 2]), ([0], [4])]:
        assert pool.fork(srcs, dsts) != 0
        after = pool.state()
        assert all(np.array_equal(after[k], before[k]) for k in before)
