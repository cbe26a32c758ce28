"""Seeded synthetic agent sessions for the forget front-end.

Draws the recorded artifact stream of a session: per turn, a few artifacts
with a type, a token span in the KV timeline, parents among earlier artifacts
and, for some, a source id they introduce (a memory field or a tool
observation bringing in outside content).  The shape follows the data flow the
paper records (Section 3.4 (a): memory/tool field -> prompt block -> model turn
-> reply/plan -> tool call -> observation -> summary write-back).

This module only draws records.  It holds none of the method: no reachability,
no boundary, no checkpoint choice.  Both the oracle (``oracle.provenance``) and
the library consume the same records.

Record: (type, turn, (span_begin, span_end), parents, sources, committed), in
append order; the type codes index ``TYPES``.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

TYPES = ("memory_field", "prompt_block", "model_turn", "reply", "plan", "tool_call",
         "observation", "summary")
MEMORY, PROMPT, MODEL, REPLY, PLAN, TOOL, OBS, SUMMARY = range(8)

Record = Tuple[int, int, Tuple[int, int], Tuple[int, ...], Tuple[int, ...], bool]


def draw_session(seed: int, n_turns: int, per_turn: int = 4, fan_in: int = 3, recent: int = 12,
                 p_inject: float = 0.15, n_source_ids: int = 8, full_state: bool = False) -> List[Record]:
    """A random session of ``n_turns`` turns.

    Per turn: 1 + Poisson(per_turn - 1) artifacts.  The first artifact of a turn
    is a prompt block, the rest are drawn from the other types.  Each artifact
    takes up to ``fan_in`` parents among the ``recent`` latest artifacts (any
    earlier turn or this one).  With probability ``p_inject`` an artifact of
    type memory_field or observation introduces a source id in
    [0, n_source_ids).  Tool calls commit an external side effect with
    probability 1/2.  With ``full_state`` every artifact also lists every
    artifact of the previous turn and every earlier artifact of its own turn as
    parents (a transition reads the whole state).  Spans are consecutive: each
    artifact occupies 1..64 tokens after the previous one.
    """
    rng = np.random.default_rng(seed)
    recs: List[Record] = []
    prev_turn: List[int] = []
    pos = 0
    for t in range(1, n_turns + 1):
        n = 1 + int(rng.poisson(max(per_turn - 1, 0)))
        this_turn: List[int] = []
        for j in range(n):
            typ = PROMPT if j == 0 else int(rng.integers(0, len(TYPES)))
            k = len(recs)
            lo = max(0, k - recent)
            n_par = int(rng.integers(0, fan_in + 1)) if k > 0 else 0
            parents = set(int(p) for p in rng.integers(lo, k, size=n_par)) if k > lo else set()
            if full_state:
                parents.update(prev_turn)
                parents.update(this_turn)
            sources: Tuple[int, ...] = ()
            if typ in (MEMORY, OBS) and rng.random() < p_inject:
                sources = (int(rng.integers(0, n_source_ids)),)
            committed = typ == TOOL and bool(rng.random() < 0.5)
            length = int(rng.integers(1, 65))
            recs.append((typ, t, (pos, pos + length), tuple(sorted(parents)), sources, committed))
            pos += length
            this_turn.append(k)
        prev_turn = this_turn
    return recs
