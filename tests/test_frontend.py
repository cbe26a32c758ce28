"""The library's forget front-end (host code behind include/pgsr.h) against the
oracle (oracle/provenance.py) on the same seeded sessions: source location,
first entry boundary, taint closure (Lemma 2), checkpoint placement and choice
(Section 3.4 (b), Algorithm 1) and the Corollary 1 counts, bit for bit (all
integer).  Host only, so these run without a GPU."""
import numpy as np
import pytest

from oracle import provenance as PV
from workloads import sessions as WS
from test_oracle_provenance import golden, golden_graph, policy

import paper_2609_04875_amd as M
from paper_2609_04875_amd import frontend as F


def lib_graph(records, extra=0):
    g = F.ProvenanceGraph(len(records) + extra, sum(len(r[3]) for r in records) + 64 * extra,
                          sum(len(r[4]) for r in records) + extra)
    g.append(records)
    return g


def oracle_graph(records):
    g = PV.ProvenanceGraph()
    for r in records:
        g.append(*r)
    return g


def lib_store(ocps):
    s = F.CheckpointStore(len(ocps) + 1)
    for c in ocps:
        s.register(c.boundary, c.token_offset, c.seq, c.env_snapshot, c.manifest)
    return s


def same_plan(lp, op):
    assert (lp.tau, lp.checkpoint, lp.boundary, lp.crop_len, lp.seq) == \
        (op.tau, op.checkpoint, op.boundary, op.crop_len, op.seq)
    assert (lp.replay_transitions, lp.minimal_transitions, lp.clean_artifacts, lp.committed_after_tau) == \
        (op.replay_transitions, op.minimal_transitions, op.clean_artifacts, op.committed_after_tau)
    assert lp.n_sources == len(op.sources) and lp.closure_size == len(op.closure)
    assert lp.closure.tolist() == list(op.closure)


def test_worked_example_through_the_abi():
    gd = golden()
    og = golden_graph(gd)
    recs = [(a["type"], a["turn"], tuple(a["span"]), tuple(a["parents"]), tuple(a["sources"]), a["committed"])
            for a in gd["artifacts"]]
    g = lib_graph(recs)
    assert g.size() == len(recs) and g.session_length() == gd["T"]
    for b, n in gd["kv_length_after"].items():
        assert g.kv_length_after(int(b)) == n
    for name, want in gd["policies"].items():
        k = int(name.rsplit("_", 1)[1]) if name.startswith("every_k_") else 1
        got = g.policy_boundaries("every_k" if name.startswith("every_k_") else name, k)
        assert got.tolist() == want, name
    for q in gd["queries"]:
        ocps = PV.checkpoints_for(og, policy(og, q["policy"]), seq=5)
        lp = F.forget_plan(g, lib_store(ocps), q["z"])
        assert lp.closure.tolist() == q["closure"] and lp.tau == q["tau"] and lp.crop_len == q["crop_len"]
        same_plan(lp, PV.forget_plan(og, ocps, q["z"]))
    for z in gd["absent"]:
        with pytest.raises(M.PgsrError) as e:
            F.forget_plan(g, lib_store(PV.checkpoints_for(og, [0])), z)
        assert e.value.code == M.ENOENT


@pytest.mark.parametrize("seed,turns,full", [(s, 40, False) for s in range(10)] +
                         [(s, 25, True) for s in range(10, 14)] + [(99, 400, False)])
def test_random_sessions_match_oracle(seed, turns, full):
    recs = WS.draw_session(seed, n_turns=turns, p_inject=0.25, n_source_ids=6, full_state=full)
    og, g = oracle_graph(recs), lib_graph(recs)
    assert g.session_length() == og.session_length()
    T = og.session_length()
    for b in range(0, T + 2):
        assert g.kv_length_after(b) == og.kv_length_after(b)
    for name in ("every_turn", "session_start", "before_injection", "every_k"):
        for k in ((1, 3, 7) if name == "every_k" else (1,)):
            assert g.policy_boundaries(name, k).tolist() == PV.policy_boundaries(og, name, k)
    rng = np.random.default_rng(seed)
    for z in range(7):
        seeds = og.locate_source(z)
        assert g.locate_source(z).tolist() == seeds
        some = sorted(set(int(x) for x in rng.integers(0, len(recs), size=3)))
        assert g.taint_closure(some).tolist() == og.taint_closure(some)
        for name in ("every_turn", "session_start", "before_injection", "every_k"):
            ocps = PV.checkpoints_for(og, PV.policy_boundaries(og, name, 5), seq=seed)
            store = lib_store(ocps)
            try:
                op = PV.forget_plan(og, ocps, z)
            except LookupError:
                with pytest.raises(M.PgsrError) as e:
                    F.forget_plan(g, store, z)
                assert e.value.code == M.ENOENT
                continue
            same_plan(F.forget_plan(g, store, z), op)


def test_checkpoint_ties_and_unsorted_registration():
    recs = WS.draw_session(7, n_turns=30, p_inject=0.3, n_source_ids=3)
    og, g = oracle_graph(recs), lib_graph(recs)
    rng = np.random.default_rng(7)
    bounds = [int(b) for b in rng.integers(0, 30, size=25)]       # unsorted, with repeats
    ocps = [PV.Checkpoint(b, og.kv_length_after(b), i, 10 * i, 20 * i) for i, b in enumerate(bounds)]
    store = lib_store(ocps)
    assert len(store) == len(ocps)
    for z in range(3):
        try:
            op = PV.forget_plan(og, ocps, z)
        except LookupError:
            continue
        lp = F.forget_plan(g, store, z)
        same_plan(lp, op)
        assert (lp.env_snapshot, lp.manifest) == (ocps[op.checkpoint].env_snapshot, ocps[op.checkpoint].manifest)


def test_monotone_under_appends():
    """Lemma 2 (i) on the library: appending in batches only grows I(z), and
    the closure of a prefix is the full closure cut at that prefix."""
    recs = WS.draw_session(11, n_turns=60, p_inject=0.3, n_source_ids=3)
    og = oracle_graph(recs)
    g = F.ProvenanceGraph(len(recs), sum(len(r[3]) for r in recs), sum(len(r[4]) for r in recs))
    prev = {z: [] for z in range(3)}
    pos = 0
    rng = np.random.default_rng(0)
    while pos < len(recs):
        n = int(rng.integers(1, 9))
        assert g.append(recs[pos:pos + n]) == pos
        pos = min(pos + n, len(recs))
        for z in range(3):
            cur = g.taint_closure(g.locate_source(z)).tolist()
            full = og.taint_closure(og.locate_source(z))
            assert set(prev[z]) <= set(cur)
            assert cur == [a for a in full if a < pos]
            prev[z] = cur


def test_invalid_appends_change_nothing_and_capacity():
    g = F.ProvenanceGraph(4, 4, 2)
    g.append([(1, 1, (0, 10), (), (), False), (2, 2, (10, 20), (0,), (5,), False)])
    bad = [(9, 2, (20, 21), (), (), False), (1, 0, (20, 21), (), (), False), (1, 2, (5, 4), (), (), False),
           (1, 2, (20, 21), (3,), (), False), (1, 1, (20, 21), (), (), False), (1, 2, (20, 21), (-1,), (), False)]
    for rec in bad:
        with pytest.raises(M.PgsrError) as e:
            g.append([(1, 2, (20, 21), (), (), False), rec])        # a good record, then a bad one
        assert e.value.code == M.EINVAL
        assert g.size() == 2
    with pytest.raises(M.PgsrError) as e:                              # 3 artifacts do not fit in 2 slots
        g.append([(1, 2, (20, 21), (), (), False)] * 3)
    assert e.value.code == M.ENOMEM and g.size() == 2
    with pytest.raises(M.PgsrError) as e:                              # 4 edges + 1 existing > 4
        g.append([(2, 3, (21, 22), (0, 1, 0, 1), (), False)])
    assert e.value.code == M.ENOMEM and g.size() == 2
    with pytest.raises(M.PgsrError) as e:                              # 2 sources + 1 existing > 2
        g.append([(0, 3, (21, 22), (), (6, 7), False)])
    assert e.value.code == M.ENOMEM and g.size() == 2
    assert g.locate_source(6).tolist() == [] and g.locate_source(5).tolist() == [1]
    s = F.CheckpointStore(1)
    s.register(0, 0)
    with pytest.raises(M.PgsrError) as e:
        s.register(1, 10)
    assert e.value.code == M.ENOMEM
    with pytest.raises(M.PgsrError) as e:
        F.CheckpointStore(2).register(-1, 0)
    assert e.value.code == M.EINVAL
    with pytest.raises(M.PgsrError):
        g.taint_closure([5])
    with pytest.raises(M.PgsrError):
        g.policy_boundaries("every_k", 0)


def test_closure_buffer_too_small_is_erange():
    import ctypes
    from paper_2609_04875_amd._native import ForgetPlanC, lib
    recs = WS.draw_session(3, n_turns=20, p_inject=0.5, n_source_ids=2, full_state=True)
    og, g = oracle_graph(recs), lib_graph(recs)
    z = next(z for z in range(2) if og.locate_source(z))
    s = lib_store(PV.checkpoints_for(og, [0]))
    p = ForgetPlanC()
    buf = np.full(1, -7, dtype=np.int64)
    rc = lib.pgsr_forget_plan_query(g._h, s._h, z, buf.ctypes.data_as(ctypes.c_void_p), 1, ctypes.byref(p))
    want = len(og.taint_closure(og.locate_source(z)))
    assert want > 1 and rc == M.ERANGE and p.closure_size == want and buf[0] == -7
