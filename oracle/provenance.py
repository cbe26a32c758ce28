"""Plain CPU oracle of the forget front-end.  TEST INFRASTRUCTURE ONLY.

Only ``tests/`` import this module.  It shares no code with
``paper_2609_04875_amd`` and never imports it.

What it follows:

* the provenance graph G of Section 3.4 (a): artifacts carrying
  (id, type, parents, source_ids, token_span, turn, committed), recorded during
  execution, append-only (the proof of Lemma 2 (i) rests on that);
* the influence set of Lemma 2: I(z) = every artifact reachable from z's
  source along recorded data-flow edges;
* the provenance queries of Algorithm 1: locate z's source artifact(s), the
  first entry boundary tau, the taint closure;
* the checkpoint set C of Section 3.4 (b): metadata only (token offset, cache
  handle, environment snapshot id, prompt manifest); the restore point c* is
  the checkpoint with the largest boundary below tau (Algorithm 1, checkpoint
  selection), and cropping the cache to its token offset restores it (Lemma 1);
* Corollary 1: replaying from c* costs T - boundary(c*) transitions, at least
  T - tau + 1, with equality when a checkpoint sits at tau - 1.

Readings where the paper is silent:
  P1 turns are 1-indexed transitions (Section 3.1); turn 0 is the initial
     state, so an artifact has turn >= 1 and a checkpoint boundary b >= 0
     names the state R_b after turn b;
  P2 an artifact may only name parents that already exist, and its turn is at
     least each parent's turn (data flows forward in time), so G is a DAG;
  P3 "source of z" = every artifact whose own source_ids contain z (where z
     enters: a memory field, a tool observation ...).  If z entered more than
     once, all entries seed the closure and tau is the earliest entry turn;
  P4 the KV length after turn b is the largest token_span end over artifacts of
     turns <= b (0 when there are none): the checkpoint at b crops to it;
  P5 several checkpoints at the same boundary: the last one registered wins;
  P6 checkpoint policies (Section 4 ablation): every_turn places boundaries
     0..T-1; session_start only 0; before_injection places 0 and t-1 for each
     turn t holding an artifact that introduces a source id; every_k places the
     multiples of k below T;
  P7 execution records artifacts as it goes, so they arrive in non-decreasing
     turn order; an artifact of an earlier turn than the last one recorded is
     rejected.
"""
from __future__ import annotations

from typing import Iterable, List, NamedTuple, Optional, Sequence, Tuple

TYPES = ("memory_field", "prompt_block", "model_turn", "reply", "plan", "tool_call",
         "observation", "summary")


class Artifact(NamedTuple):
    id: int
    type: int
    turn: int
    span: Tuple[int, int]
    parents: Tuple[int, ...]
    sources: frozenset
    committed: bool


class ProvenanceGraph:
    """Artifact-level data flow (Section 3.4 (a)), append-only."""

    def __init__(self):
        self.artifacts: List[Artifact] = []

    def append(self, type: int, turn: int, span: Tuple[int, int], parents: Sequence[int] = (),
               sources: Iterable[int] = (), committed: bool = False) -> int:
        """Record one artifact; returns its id (ids are 0, 1, 2, ... in order).
        Invalid records raise ValueError and leave the graph unchanged (P1, P2, P7)."""
        parents = tuple(int(p) for p in parents)
        if not 0 <= type < len(TYPES):
            raise ValueError("unknown artifact type")
        if turn < 1:
            raise ValueError("turns start at 1")
        if self.artifacts and turn < self.artifacts[-1].turn:
            raise ValueError("artifacts arrive in turn order")
        if span[0] < 0 or span[1] < span[0]:
            raise ValueError("bad token span")
        for p in parents:
            if not 0 <= p < len(self.artifacts):
                raise ValueError("parent does not exist")
            if self.artifacts[p].turn > turn:
                raise ValueError("data cannot flow back in time")
        aid = len(self.artifacts)
        self.artifacts.append(Artifact(aid, int(type), int(turn), (int(span[0]), int(span[1])), parents,
                                       frozenset(int(s) for s in sources), bool(committed)))
        return aid

    def session_length(self) -> int:
        """T: the last turn recorded (0 for an empty graph)."""
        return max((a.turn for a in self.artifacts), default=0)

    def locate_source(self, z: int) -> List[int]:
        """Artifacts where z enters (P3), ascending ids."""
        return [a.id for a in self.artifacts if z in a.sources]

    def first_entry(self, seeds: Sequence[int]) -> int:
        """tau: the earliest turn at which z is part of the runtime."""
        return min(self.artifacts[s].turn for s in seeds)

    def taint_closure(self, seeds: Sequence[int]) -> List[int]:
        """I(z) of Lemma 2: the seeds and everything reachable from them.
        Brute-force fixpoint: a child of a tainted artifact is tainted; repeat
        until nothing changes."""
        tainted = set(seeds)
        changed = True
        while changed:
            changed = False
            for a in self.artifacts:
                if a.id not in tainted and any(p in tainted for p in a.parents):
                    tainted.add(a.id)
                    changed = True
        return sorted(tainted)

    def certified_clean(self, tau: int) -> List[int]:
        """Lemma 2 (ii): the artifacts of turns before tau."""
        return [a.id for a in self.artifacts if a.turn < tau]

    def kv_length_after(self, b: int) -> int:
        """Tokens in the cache once turn b is done (P4)."""
        return max((a.span[1] for a in self.artifacts if a.turn <= b), default=0)


class Checkpoint(NamedTuple):
    """Section 3.4 (b): metadata only, no tensor copies."""
    boundary: int
    token_offset: int
    seq: int
    env_snapshot: int
    manifest: int


def policy_boundaries(graph: ProvenanceGraph, policy: str, k: int = 1) -> List[int]:
    """Checkpoint boundaries a placement policy yields for a recorded session (P6)."""
    T = graph.session_length()
    if policy == "every_turn":
        return list(range(T))
    if policy == "session_start":
        return [0]
    if policy == "before_injection":
        inj = sorted({a.turn - 1 for a in graph.artifacts if a.sources})
        return sorted({0, *inj})
    if policy == "every_k":
        return list(range(0, T, k))
    raise ValueError(policy)


def checkpoints_for(graph: ProvenanceGraph, boundaries: Sequence[int], seq: int = 0) -> List[Checkpoint]:
    """Checkpoints at the given boundaries, token offsets from the graph (P4)."""
    return [Checkpoint(b, graph.kv_length_after(b), seq, 1000 + b, 2000 + b) for b in boundaries]


def select_checkpoint(checkpoints: Sequence[Checkpoint], tau: int) -> Optional[int]:
    """c* = argmax {c : boundary(c) < tau}; the index in registration order, or
    None when no checkpoint lies before tau (P5: the last registered wins ties)."""
    best = None
    for i, c in enumerate(checkpoints):
        if c.boundary < tau and (best is None or c.boundary >= checkpoints[best].boundary):
            best = i
    return best


class ForgetPlan(NamedTuple):
    sources: Tuple[int, ...]        # where z entered
    tau: int                        # first entry boundary
    closure: Tuple[int, ...]        # I(z), ascending ids
    checkpoint: int                 # index of c*
    boundary: int                   # boundary(c*)
    crop_len: int                   # tokens kept by the crop (token offset of c*)
    seq: int                        # cache handle of c*
    replay_transitions: int         # T - boundary(c*)
    minimal_transitions: int        # T - tau + 1 (Corollary 1)
    clean_artifacts: int            # |{a : turn(a) < tau}| (Lemma 2 (ii))
    committed_after_tau: int        # artifacts at turns >= tau with committed side effects


def forget_plan(graph: ProvenanceGraph, checkpoints: Sequence[Checkpoint], z: int) -> ForgetPlan:
    """Algorithm 1's provenance queries and checkpoint selection for target z.
    Raises LookupError when z is not in the graph or no checkpoint precedes tau."""
    seeds = graph.locate_source(z)
    if not seeds:
        raise LookupError("z never entered the session")
    tau = graph.first_entry(seeds)
    closure = graph.taint_closure(seeds)
    ci = select_checkpoint(checkpoints, tau)
    if ci is None:
        raise LookupError("no checkpoint before tau")
    c = checkpoints[ci]
    T = graph.session_length()
    return ForgetPlan(tuple(seeds), tau, tuple(closure), ci, c.boundary, c.token_offset, c.seq,
                      T - c.boundary, T - tau + 1, len(graph.certified_clean(tau)),
                      sum(1 for a in graph.artifacts if a.turn >= tau and a.committed))
