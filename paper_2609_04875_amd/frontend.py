"""Forget front-end: the provenance graph, checkpoint store and forget query
of ``include/pgsr.h`` (Section 3.4 (a)/(b); Lemma 2; Algorithm 1, the steps
before the restore).  Argument marshalling only; the work runs in the
library's host code."""
from __future__ import annotations

import ctypes
from typing import NamedTuple, Sequence

import numpy as np

from ._native import ForgetPlanC, PgsrError, check, lib

POLICIES = {"every_turn": 0, "session_start": 1, "before_injection": 2, "every_k": 3}


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p) if a.size else None


def _ids(call, *args) -> np.ndarray:
    """Two-pass helper for the (out, capacity, n_out) convention."""
    n = ctypes.c_int64()
    check(call(*args, None, 0, ctypes.byref(n)))
    out = np.empty(max(n.value, 1), dtype=np.int64)
    check(call(*args, out.ctypes.data_as(ctypes.c_void_p), out.size, ctypes.byref(n)))
    return out[:n.value]


class ProvenanceGraph:
    """Append-only artifact graph with fixed capacities (host memory)."""

    def __init__(self, max_artifacts: int, max_edges: int, max_sources: int):
        h = ctypes.c_void_p()
        check(lib.pgsr_graph_create(max_artifacts, max_edges, max_sources, ctypes.byref(h)))
        self._h = h

    def close(self) -> None:
        if self._h:
            lib.pgsr_graph_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def append(self, records: Sequence) -> int:
        """Record (type, turn, (begin, end), parents, sources, committed) tuples;
        returns the first new id.  Raises PgsrError (nothing recorded) on a bad
        record or when the capacity is exceeded."""
        n = len(records)
        types = np.array([r[0] for r in records], dtype=np.int32)
        turns = np.array([r[1] for r in records], dtype=np.int32)
        sb = np.array([r[2][0] for r in records], dtype=np.int64)
        se = np.array([r[2][1] for r in records], dtype=np.int64)
        poff = np.zeros(n + 1, dtype=np.int64)
        soff = np.zeros(n + 1, dtype=np.int64)
        poff[1:] = np.cumsum([len(r[3]) for r in records]) if n else []
        soff[1:] = np.cumsum([len(r[4]) for r in records]) if n else []
        par = np.array([p for r in records for p in r[3]], dtype=np.int64)
        src = np.array([z for r in records for z in r[4]], dtype=np.int64)
        com = np.array([1 if r[5] else 0 for r in records], dtype=np.uint8)
        first = ctypes.c_int64(-1)
        check(lib.pgsr_graph_append(self._h, n, _ptr(types), _ptr(turns), _ptr(sb), _ptr(se),
                                    _ptr(poff), _ptr(par), _ptr(soff), _ptr(src), _ptr(com),
                                    ctypes.byref(first)))
        return first.value

    def size(self) -> int:
        n = ctypes.c_int64()
        check(lib.pgsr_graph_size(self._h, ctypes.byref(n)))
        return n.value

    def session_length(self) -> int:
        t = ctypes.c_int64()
        check(lib.pgsr_graph_session_length(self._h, ctypes.byref(t)))
        return t.value

    def kv_length_after(self, b: int) -> int:
        n = ctypes.c_int64()
        check(lib.pgsr_graph_kv_length_after(self._h, b, ctypes.byref(n)))
        return n.value

    def locate_source(self, z: int) -> np.ndarray:
        return _ids(lib.pgsr_graph_locate_source, self._h, z)

    def taint_closure(self, seeds: Sequence[int]) -> np.ndarray:
        s = np.asarray(seeds, dtype=np.int64)
        return _ids(lib.pgsr_graph_taint_closure, self._h, _ptr(s), s.size)

    def policy_boundaries(self, policy: str, k: int = 1) -> np.ndarray:
        return _ids(lib.pgsr_graph_policy_boundaries, self._h, POLICIES[policy], k)


class CheckpointStore:
    """Metadata-only checkpoints (Section 3.4 (b))."""

    def __init__(self, capacity: int):
        h = ctypes.c_void_p()
        check(lib.pgsr_ckpt_create(capacity, ctypes.byref(h)))
        self._h = h

    def close(self) -> None:
        if self._h:
            lib.pgsr_ckpt_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def register(self, boundary: int, token_offset: int, seq: int = 0, env_snapshot: int = 0,
                 manifest: int = 0) -> None:
        check(lib.pgsr_ckpt_register(self._h, boundary, token_offset, seq, env_snapshot, manifest))

    def __len__(self) -> int:
        n = ctypes.c_int64()
        check(lib.pgsr_ckpt_count(self._h, ctypes.byref(n)))
        return n.value


class ForgetPlan(NamedTuple):
    tau: int
    checkpoint: int
    boundary: int
    crop_len: int
    seq: int
    env_snapshot: int
    manifest: int
    replay_transitions: int
    minimal_transitions: int
    n_sources: int
    closure_size: int
    clean_artifacts: int
    committed_after_tau: int
    closure: np.ndarray


def forget_plan(graph: ProvenanceGraph, store: CheckpointStore, z: int, with_closure: bool = True) -> ForgetPlan:
    """Algorithm 1's provenance queries and restore point for target z.
    Raises PgsrError with code ENOENT when z never entered or no checkpoint
    precedes tau."""
    p = ForgetPlanC()
    check(lib.pgsr_forget_plan_query(graph._h, store._h, z, None, 0, ctypes.byref(p)))
    clo = np.empty(0, dtype=np.int64)
    if with_closure and p.closure_size:
        clo = np.empty(p.closure_size, dtype=np.int64)
        check(lib.pgsr_forget_plan_query(graph._h, store._h, z, clo.ctypes.data_as(ctypes.c_void_p),
                                         clo.size, ctypes.byref(p)))
    return ForgetPlan(*[getattr(p, f) for f, _ in ForgetPlanC._fields_], closure=clo)


__all__ = ["ProvenanceGraph", "CheckpointStore", "ForgetPlan", "forget_plan", "POLICIES", "PgsrError"]
