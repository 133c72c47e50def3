"""CPU oracle for SMORE's query sampler (arXiv 2110.14890).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  Nothing here imports the GPU library,
and the GPU library never imports this package.

- ``liboracle.so`` (oracle.c, plain C): Philox4x32-10, adjacency, exhaustive
  answer sets, reverse directional sampling, negatives by membership in the
  exhaustive answer set, and a generic bidirectional checker.
- ``brute``: pure-Python evaluation of the first-order formulas of the
  paper's query definition by enumerating every variable assignment.
- ``cuts``: brute-force enumeration of node cuts and the cost objective of
  the optimal-scheduling equation.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")


def build(force: bool = True) -> str:
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, src])
        os.replace(tmp, _SO)
    return _SO


class _Args(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_neg", ctypes.c_int32),
                ("pos_tries", ctypes.c_int32), ("neg_tries", ctypes.c_int32),
                ("max_fanout", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("query_offset", ctypes.c_uint64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build(force=False)
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        L.oracle_philox.argtypes = [P, P, P]
        L.oracle_pick.restype = ctypes.c_uint64
        L.oracle_pick.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.oracle_draw.restype = ctypes.c_uint64
        L.oracle_draw.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                  ctypes.c_uint32, ctypes.c_uint32]
        L.oracle_graph_build.restype = P
        L.oracle_graph_build.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int, ctypes.c_int]
        L.oracle_graph_free.argtypes = [P]
        L.oracle_graph_stats.argtypes = [P, P]
        L.oracle_graph_edges.restype = ctypes.c_int64
        L.oracle_graph_edges.argtypes = [P, ctypes.c_int, ctypes.c_int32, P, P]
        L.oracle_graph_dump.restype = ctypes.c_int64
        L.oracle_graph_dump.argtypes = [P, ctypes.c_int, P, P, P]
        L.oracle_graph_active_in.restype = ctypes.c_int64
        L.oracle_graph_active_in.argtypes = [P, P]
        L.oracle_sample.argtypes = [P, ctypes.c_int, ctypes.POINTER(_Args), P, P, P, P, P, P, P,
                                    ctypes.c_int]
        L.oracle_sample_shared.argtypes = [P, ctypes.c_int, ctypes.POINTER(_Args), P, P, P, P, P, P,
                                           P, P, ctypes.c_int]
        L.oracle_verify.argtypes = [P, ctypes.c_int, ctypes.c_int32, ctypes.c_int32, P, P, P, P, P,
                                    ctypes.c_int]
        L.oracle_answer_set.restype = ctypes.c_int64
        L.oracle_answer_set.argtypes = [P, ctypes.c_int, P, P, P, ctypes.c_int64]
        L.oracle_bidir_check.argtypes = [P, ctypes.c_int, P, P, ctypes.c_uint32, ctypes.c_int32, P]
        L.oracle_verify_lines_batch.argtypes = [P, ctypes.c_int, ctypes.c_int32, P, P, P,
                                                 ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64,
                                                 ctypes.c_int32, P, ctypes.c_int]
        L.oracle_set_proj_mode.argtypes = [ctypes.c_int]
        L.oracle_type_plan.argtypes = [ctypes.c_int, P, P, P, P]
        _lib = L
    return _lib


def philox(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def pick(u: int, n: int) -> int:
    return int(lib().oracle_pick(u, n))


def draw(seed: int, tag: int, qid: int, t: int, j: int) -> int:
    return int(lib().oracle_draw(seed, tag, qid, t, j))


def set_proj_mode(mode: int) -> None:
    lib().oracle_set_proj_mode(mode)


def type_plan(qtype: str):
    """(op, child[n,3], slot, root) of the oracle's computation plan."""
    op = np.zeros(8, np.int32)
    ch = np.zeros(24, np.int32)
    sl = np.zeros(8, np.int32)
    root = np.zeros(1, np.int32)
    n = lib().oracle_type_plan(TYPES.index(qtype), op.ctypes.data, ch.ctypes.data,
                               sl.ctypes.data, root.ctypes.data)
    return op[:n].copy(), ch[:3 * n].reshape(n, 3).copy(), sl[:n].copy(), int(root[0])


class Graph:
    """Oracle adjacency built from int32 [E,3] triples."""

    def __init__(self, triples, n_entities: int, n_relations: int, add_inverse: bool = False,
                 threads: int = 0):
        tr = np.ascontiguousarray(triples, dtype=np.int32).reshape(-1, 3)
        self._h = lib().oracle_graph_build(tr.ctypes.data if len(tr) else None, len(tr),
                                           n_entities, n_relations, int(add_inverse), threads)
        if not self._h:
            raise ValueError("oracle_graph_build rejected the triples")
        st = np.zeros(9, np.int64)
        lib().oracle_graph_stats(self._h, st.ctypes.data)
        (self.V, self.R, self.E, self.S_fwd, self.S_rev, self.n_active, self.max_out,
         self.max_in, self.max_seg) = [int(x) for x in st]

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().oracle_graph_free(h)
            self._h = None

    def edges(self, v: int, reverse: bool = False):
        n = lib().oracle_graph_edges(self._h, int(reverse), v, None, None)
        rel = np.zeros(max(n, 1), np.int32)
        nbr = np.zeros(max(n, 1), np.int32)
        lib().oracle_graph_edges(self._h, int(reverse), v, rel.ctypes.data, nbr.ctypes.data)
        return rel[:n], nbr[:n]

    def dump(self, reverse: bool = False):
        """(entity, relation, neighbour) of every edge in canonical order."""
        n = max(self.E, 1)
        e, r, o = np.zeros(n, np.int32), np.zeros(n, np.int32), np.zeros(n, np.int32)
        lib().oracle_graph_dump(self._h, int(reverse), e.ctypes.data, r.ctypes.data, o.ctypes.data)
        return e[:self.E], r[:self.E], o[:self.E]

    def active_in(self):
        out = np.zeros(max(self.n_active, 1), np.int32)
        lib().oracle_graph_active_in(self._h, out.ctypes.data)
        return out[:self.n_active]

    def answer_set(self, qtype: str, anchors, relations):
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(relations, np.int32)
        n = lib().oracle_answer_set(self._h, TYPES.index(qtype), a.ctypes.data, r.ctypes.data,
                                    None, 0)
        if n < 0:
            raise ValueError("bad query")
        out = np.zeros(max(n, 1), np.int32)
        lib().oracle_answer_set(self._h, TYPES.index(qtype), a.ctypes.data, r.ctypes.data,
                                out.ctypes.data, n)
        return out[:n]

    def bidir_check(self, qtype: str, anchors, relations, cut_mask: int, c: int):
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(relations, np.int32)
        counts = np.zeros(2, np.int64)
        rc = lib().oracle_bidir_check(self._h, TYPES.index(qtype), a.ctypes.data, r.ctypes.data,
                                      cut_mask, c, counts.ctypes.data)
        return rc, int(counts[0]), int(counts[1])

    def sample(self, qtype: str, batch: int, n_neg: int, seed: int = 0, query_offset: int = 0,
               pos_tries: int = 64, neg_tries: int | None = None, max_fanout: int = 0,
               threads: int = 0):
        if neg_tries is None:
            neg_tries = 4 * n_neg
        a = _Args(batch, n_neg, pos_tries, neg_tries, max_fanout, seed, query_offset)
        out = {
            "anchors": np.zeros((batch, 3), np.int32),
            "relations": np.zeros((batch, 3), np.int32),
            "positive": np.zeros(batch, np.int32),
            "negatives": np.zeros((batch, n_neg), np.int32),
            "n_valid": np.zeros(batch, np.int32),
            "pos_attempts": np.zeros(batch, np.int32),
            "neg_draws": np.zeros(batch, np.int32),
        }
        rc = lib().oracle_sample(self._h, TYPES.index(qtype), ctypes.byref(a),
                                 out["anchors"].ctypes.data, out["relations"].ctypes.data,
                                 out["positive"].ctypes.data, out["negatives"].ctypes.data,
                                 out["n_valid"].ctypes.data, out["pos_attempts"].ctypes.data,
                                 out["neg_draws"].ctypes.data, threads)
        if rc != 0:
            raise ValueError("oracle_sample rejected its arguments")
        return out

    def verify(self, qtype: str, anchors, relations, candidates, threads: int = 0):
        """Mask of the candidates [batch, n] that are entities outside A_q."""
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(relations, np.int32)
        c = np.ascontiguousarray(candidates, np.int32)
        batch, n = c.shape
        mask = np.zeros((batch, (n + 31) // 32), np.uint32)
        nv = np.zeros(batch, np.int32)
        rc = lib().oracle_verify(self._h, TYPES.index(qtype), batch, n, a.ctypes.data, r.ctypes.data,
                                 c.ctypes.data, mask.ctypes.data, nv.ctypes.data, threads)
        if rc != 0:
            raise ValueError("oracle_verify rejected its arguments")
        return {"mask": mask, "n_valid": nv}

    def verify_lines(self, qtype: str, anchors, relations, positive, cut_mask: int, seed: int,
                     query_offset: int, n_draws: int, threads: int = 0) -> np.ndarray:
        """Distinct 64-byte lines a bidirectional check reads per query
        (oracle_verify_lines_batch): int64 [batch, 3] = first-pass part,
        long-list part, both."""
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(relations, np.int32)
        p = np.ascontiguousarray(positive, np.int32)
        out = np.zeros((len(p), 3), np.int64)
        rc = lib().oracle_verify_lines_batch(self._h, TYPES.index(qtype), len(p), a.ctypes.data,
                                             r.ctypes.data, p.ctypes.data, cut_mask, seed,
                                             query_offset, n_draws, out.ctypes.data, threads)
        if rc != 0:
            raise ValueError("oracle_verify_lines rejected its arguments")
        return out

    def sample_shared(self, qtype: str, batch: int, n_shared: int, seed: int = 0,
                      query_offset: int = 0, pos_tries: int = 64, neg_tries: int | None = None,
                      max_fanout: int = 0, threads: int = 0):
        """Minibatch with one shared candidate set (oracle_sample_shared)."""
        if neg_tries is None:
            neg_tries = 4 * n_shared
        a = _Args(batch, n_shared, pos_tries, neg_tries, max_fanout, seed, query_offset)
        words = (n_shared + 31) // 32
        out = {
            "anchors": np.zeros((batch, 3), np.int32),
            "relations": np.zeros((batch, 3), np.int32),
            "positive": np.zeros(batch, np.int32),
            "pos_attempts": np.zeros(batch, np.int32),
            "shared": np.zeros(n_shared, np.int32),
            "n_shared": np.zeros(1, np.int32),
            "mask": np.zeros((batch, words), np.uint32),
            "n_valid": np.zeros(batch, np.int32),
        }
        rc = lib().oracle_sample_shared(self._h, TYPES.index(qtype), ctypes.byref(a),
                                        *[out[k].ctypes.data for k in
                                          ("anchors", "relations", "positive", "pos_attempts",
                                           "shared", "n_shared", "mask", "n_valid")], threads)
        if rc != 0:
            raise ValueError("oracle_sample_shared rejected its arguments")
        return out
