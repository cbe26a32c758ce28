"""The replay entry point that allocates nothing (pgsr_replay_prefill_static),
called through the C ABI, against pgsr_replay_prefill on a pool whose
workspace has the same size: two calls in a row, the second smaller (a split
prefill, then a decode step that leaves fewer partials over the first call's),
equal bit for bit and within the bf16 tolerance of the oracle; a size past the
static scratch is rejected and changes nothing."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import assert_close, dev, log, make_pool, oracle_suffix

pytestmark = pytest.mark.gpu

GEOM = W.AttnGeometry(32, 8, 128)
SCALE = 128 ** -0.5


def _blocks(n, B=16):
    return -(-n // B)


def test_static_scratch_replay_equals_workspace_replay():
    from paper_2609_04875_amd import ERANGE, workspace_bytes
    from paper_2609_04875_amd import _native as N
    rng = np.random.default_rng(41)
    P, S1, S2 = 3001, 256, 4
    ep = W.draw_episode(rng, GEOM, "bf16", P, S1, P + 40)
    ws = workspace_bytes(GEOM.n_q_heads, GEOM.head_dim, S1, 8)
    assert 0 < ws <= N.STATIC_SCRATCH_BYTES
    log(f"no-alloc replay: P={P}, calls of {S1} then {S2} tokens, scratch {ws} bytes")
    nb = _blocks(P + 40) + _blocks(P + S1) + 8
    ref_pool = make_pool(GEOM, "bf16", nb, 1, 256, split_q=S1, max_splits=8)
    assert ref_pool.workspace.numel() == ws
    pool = make_pool(GEOM, "bf16", nb, 1, 256)          # no workspace of its own
    for p in (ref_pool, pool):
        cq, ck, cv = (dev(ep.contaminated(x), "bf16") for x in ("q", "k", "v"))
        assert p.replay(0, [0], [ep.t_contaminated], cq, ck, cv, torch.empty_like(cq), SCALE) == 0
        assert p.crop([0], [P]) == 0
    for S in (S1, S2):
        q, k, v = (dev(getattr(ep, x)[P:P + S], "bf16") for x in ("q", "k", "v"))
        o_ref = torch.full_like(q, float("nan"))
        o = torch.full_like(q, float("nan"))
        assert ref_pool.replay(0, [0], [S], q, k, v, o_ref, SCALE, commit=False) == 0
        assert pool.replay_static(0, [0], [S], q, k, v, o, SCALE, ws, commit=False) == 0
        torch.cuda.synchronize()
        assert torch.equal(o, o_ref), f"S={S}"
        sub = W.Episode("bf16", P, S, P, ep.q[:P + S], ep.k[:P + S], ep.v[:P + S], ep.cq, ep.ck, ep.cv)
        assert_close(o.float().cpu().numpy(), oracle_suffix(sub, SCALE), "bf16", f"static scratch, S={S}")
        # the split / decode path really ran: an unsplit replay rounds differently
        plain = make_pool(GEOM, "bf16", nb, 1, 256)
        cq, ck, cv = (dev(ep.contaminated(x), "bf16") for x in ("q", "k", "v"))
        assert plain.replay(0, [0], [ep.t_contaminated], cq, ck, cv, torch.empty_like(cq), SCALE) == 0
        assert plain.crop([0], [P]) == 0
        o_plain = torch.empty_like(q)
        assert plain.replay(0, [0], [S], q, k, v, o_plain, SCALE, commit=False) == 0
        assert not torch.equal(o_plain, o), f"S={S}: no split happened"
        del plain
    # a size past the static scratch: rejected, nothing changes
    before = pool.state()
    q, k, v = (dev(getattr(ep, x)[P:P + S2], "bf16") for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    assert pool.replay_static(0, [0], [S2], q, k, v, o, SCALE, N.STATIC_SCRATCH_BYTES + 1) == ERANGE
    assert b"exceeds the static scratch" in N.lib.pgsr_last_error()
    after = pool.state()
    for key in before:
        assert np.array_equal(np.asarray(before[key]), np.asarray(after[key])), key
