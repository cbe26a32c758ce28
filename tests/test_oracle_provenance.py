"""Pins of the forget front-end oracle (oracle/provenance.py) against what the
paper and plain graph theory fix: a hand-worked session (Section 3.4, Lemma 2,
Algorithm 1, Corollary 1), transitive closure by boolean matrix powers, the
monotonicity of Lemma 2 (i), the certifiable boundary of Lemma 2 (ii), and
checkpoint choice by exhaustive search."""
import json
import os

import numpy as np
import pytest

from oracle import provenance as PV
from workloads import sessions as WS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "provenance_worked_example.json")


def build(records):
    g = PV.ProvenanceGraph()
    for typ, turn, span, parents, sources, committed in records:
        g.append(typ, turn, span, parents, sources, committed)
    return g


def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def golden_graph(gd):
    recs = [(a["type"], a["turn"], tuple(a["span"]), tuple(a["parents"]), tuple(a["sources"]), a["committed"])
            for a in gd["artifacts"]]
    return build(recs)


def policy(g, name):
    if name.startswith("every_k_"):
        return PV.policy_boundaries(g, "every_k", int(name.rsplit("_", 1)[1]))
    return PV.policy_boundaries(g, name)


def test_worked_example():
    gd = golden()
    g = golden_graph(gd)
    assert PV.TYPES == tuple(gd["types"]) == WS.TYPES
    assert g.session_length() == gd["T"]
    for b, n in gd["kv_length_after"].items():
        assert g.kv_length_after(int(b)) == n
    for name, want in gd["policies"].items():
        assert policy(g, name) == want, name
    for q in gd["queries"]:
        cps = PV.checkpoints_for(g, policy(g, q["policy"]), seq=5)
        p = PV.forget_plan(g, cps, q["z"])
        got = {"sources": list(p.sources), "tau": p.tau, "closure": list(p.closure), "boundary": p.boundary,
               "crop_len": p.crop_len, "replay_transitions": p.replay_transitions,
               "minimal_transitions": p.minimal_transitions, "clean_artifacts": p.clean_artifacts,
               "committed_after_tau": p.committed_after_tau}
        assert got == {k: q[k] for k in got}, (q["z"], q["policy"])
        assert p.seq == 5
    for z in gd["absent"]:
        with pytest.raises(LookupError):
            PV.forget_plan(g, PV.checkpoints_for(g, [0]), z)


def closure_by_matrix(records, seeds):
    """Reachability by boolean matrix powers: R <- R or R A until fixed."""
    n = len(records)
    adj = np.zeros((n, n), dtype=bool)
    for c, rec in enumerate(records):
        for p in rec[3]:
            adj[p, c] = True
    reach = np.eye(n, dtype=bool)
    while True:
        nxt = reach | ((reach.astype(np.int64) @ adj.astype(np.int64)) > 0)
        if (nxt == reach).all():
            break
        reach = nxt
    return sorted(set(np.nonzero(reach[list(seeds)].any(axis=0))[0].tolist())) if seeds else []


@pytest.mark.parametrize("seed", range(12))
def test_closure_matches_matrix_reachability(seed):
    recs = WS.draw_session(seed, n_turns=20, per_turn=3, p_inject=0.3, n_source_ids=4)
    g = build(recs)
    for z in range(4):
        seeds = g.locate_source(z)
        assert seeds == [i for i, r in enumerate(recs) if z in r[4]]
        assert g.taint_closure(seeds) == closure_by_matrix(recs, seeds)


@pytest.mark.parametrize("seed", range(6))
def test_lemma2_monotone_in_appends(seed):
    """Lemma 2 (i): the influence set only grows as execution appends."""
    recs = WS.draw_session(100 + seed, n_turns=25, p_inject=0.3, n_source_ids=3)
    g_full = build(recs)
    for z in range(3):
        prev = []
        for n in range(1, len(recs) + 1, 3):
            g = build(recs[:n])
            cur = g.taint_closure(g.locate_source(z))
            assert set(prev) <= set(cur)
            full = g_full.taint_closure(g_full.locate_source(z))
            assert cur == [a for a in full if a < n]      # later appends never change earlier reach
            prev = cur


@pytest.mark.parametrize("seed", range(6))
def test_lemma2_certified_boundary(seed):
    """Lemma 2 (ii): the closure lies at turns >= tau, disjoint from the clean
    prefix; when every transition reads the whole state the closure is every
    artifact after turn tau plus those of turn tau from z's first entry on."""
    for full_state in (False, True):
        recs = WS.draw_session(200 + seed, n_turns=15, p_inject=0.4, n_source_ids=3, full_state=full_state)
        g = build(recs)
        for z in range(3):
            seeds = g.locate_source(z)
            if not seeds:
                continue
            tau = g.first_entry(seeds)
            clo = set(g.taint_closure(seeds))
            clean = set(g.certified_clean(tau))
            assert all(g.artifacts[a].turn >= tau for a in clo)
            assert not clo & clean
            if full_state:
                first = min(s for s in seeds if g.artifacts[s].turn == tau)
                assert clo == {a.id for a in g.artifacts if a.turn > tau or (a.turn == tau and a.id >= first)}


@pytest.mark.parametrize("seed", range(8))
def test_checkpoint_choice_exhaustive(seed):
    """c* = the largest boundary below tau (the last registered among equals);
    Corollary 1: replay >= T - tau + 1, with equality for every_turn."""
    rng = np.random.default_rng(300 + seed)
    recs = WS.draw_session(300 + seed, n_turns=30, p_inject=0.3, n_source_ids=4)
    g = build(recs)
    T = g.session_length()
    bounds = [int(b) for b in rng.integers(0, T, size=7)]
    cps = PV.checkpoints_for(g, bounds)
    for tau in range(0, T + 2):
        below = [i for i, c in enumerate(cps) if c.boundary < tau]
        want = max(below, key=lambda i: (cps[i].boundary, i)) if below else None
        assert PV.select_checkpoint(cps, tau) == want
    for z in range(4):
        seeds = g.locate_source(z)
        if not seeds:
            continue
        every = PV.forget_plan(g, PV.checkpoints_for(g, PV.policy_boundaries(g, "every_turn")), z)
        assert every.boundary == every.tau - 1
        assert every.replay_transitions == every.minimal_transitions == T - every.tau + 1
        start = PV.forget_plan(g, PV.checkpoints_for(g, [0]), z)
        assert start.replay_transitions == T and start.crop_len == 0
        for name in ("before_injection", "every_k"):
            p = PV.forget_plan(g, PV.checkpoints_for(g, PV.policy_boundaries(g, name, 4)), z)
            assert p.boundary < p.tau
            assert p.replay_transitions >= p.minimal_transitions
            assert p.crop_len == g.kv_length_after(p.boundary)
        # before_injection always holds a checkpoint at tau - 1 (z enters at an injection)
        inj = PV.forget_plan(g, PV.checkpoints_for(g, PV.policy_boundaries(g, "before_injection")), z)
        assert inj.boundary == inj.tau - 1


def test_invalid_appends_change_nothing():
    g = PV.ProvenanceGraph()
    g.append(1, 1, (0, 10))
    g.append(2, 2, (10, 20), parents=[0])
    before = list(g.artifacts)
    for bad in [dict(type=9, turn=2, span=(20, 21)), dict(type=1, turn=0, span=(20, 21)),
                dict(type=1, turn=2, span=(5, 4)), dict(type=1, turn=2, span=(20, 21), parents=[2]),
                dict(type=1, turn=1, span=(20, 21), parents=[1]), dict(type=1, turn=1, span=(20, 21))]:
        with pytest.raises(ValueError):
            g.append(**bad)
        assert g.artifacts == before
    assert PV.ProvenanceGraph().session_length() == 0
    with pytest.raises(LookupError):
        PV.forget_plan(g, [], 1)
    g.append(0, 3, (20, 30), sources=[4])
    with pytest.raises(LookupError):                      # no checkpoint below tau = 3
        PV.forget_plan(g, [PV.Checkpoint(3, 0, 0, 0, 0)], 4)
