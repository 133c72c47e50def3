"""Seeded synthetic knowledge graphs shaped like the paper's datasets.

Inputs only: this module holds none of the sampling method's arithmetic.
Both the CPU oracle and the GPU library take the triples it returns.

The five configurations stand in for the knowledge graphs of the paper's
statistics table (FB15k-237, FB400k, ogbl-wikikg2, Freebase); those datasets
are not used.  Entity and relation ids are drawn as ranks from rank-Zipf laws
(P(rank k) ~ k^-s) or uniformly, and mapped to ids by seeded permutations;
the graph is the first E distinct triples of the candidate stream (see
kgsynth.c for the exact recipe).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libkgsynth.so")


@dataclass(frozen=True)
class KGConfig:
    name: str
    n_entities: int
    n_relations: int
    n_triples: int
    head_zipf: bool
    head_s: float
    tail_zipf: bool
    tail_s: float
    rel_zipf: bool
    rel_s: float
    shared_perm: bool
    deg_cap: int
    add_inverse: bool
    query_types: tuple
    batch: int
    n_neg: int
    seed: int = 0
    graph_seed: int = 0
    extra: dict = field(default_factory=dict)


ALL_TYPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up")

CONFIGS = {
    # tiny uniform graph; reverse edges added at graph build
    "tiny": KGConfig("tiny", 1_000, 20, 10_000, False, 0.0, False, 0.0, False, 0.0,
                     False, 0, True, ("1p", "2p", "3p"), 1024, 32),
    # FB15k-237-shaped: head Zipf(1.1), tail uniform, relation Zipf(1.0)
    "fb15k237": KGConfig("fb15k237", 15_000, 237, 310_000, True, 1.1, False, 0.0, True, 1.0,
                         False, 0, False, ALL_TYPES, 512, 128),
    # FB400k-shaped: Zipf(1.2) endpoints sharing one permutation, degrees capped at 50,000
    "fb400k": KGConfig("fb400k", 400_000, 900, 2_100_000, True, 1.2, True, 1.2, True, 1.0,
                       True, 50_000, False, ("2p", "3p", "ip", "pi"), 4096, 256),
    # ogbl-wikikg2-shaped: Zipf(1.2) endpoints sharing one permutation
    "wikikg2": KGConfig("wikikg2", 2_500_000, 535, 17_000_000, True, 1.2, True, 1.2, True, 1.0,
                        True, 0, False, ALL_TYPES, 8192, 256, extra={"overdraw": 2.6}),
    # Freebase-shaped: 86M entities, Zipf(1.3) endpoints sharing one permutation
    "freebase": KGConfig("freebase", 86_000_000, 14_800, 338_000_000, True, 1.3, True, 1.3,
                         True, 1.0, True, 0, False, ("3p", "ip", "pi"), 16384, 512,
                         extra={"overdraw": 5.2}),
}


def build(force: bool = True) -> str:
    """Compile the generator with gcc (OpenMP)."""
    src = os.path.join(_HERE, "kgsynth.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O3", "-march=x86-64-v2", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, src, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build(force=False)
        lib = ctypes.CDLL(_SO)
        lib.kgs_generate.restype = ctypes.c_int64
        lib.kgs_generate.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_double,
                                     ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_int64,
                                     ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p,
                                     ctypes.c_int]
        _lib = lib
    return _lib


def generate_raw(n_entities, n_relations, n_triples, *, head_zipf=False, head_s=0.0,
                 tail_zipf=False, tail_s=0.0, rel_zipf=False, rel_s=0.0, shared_perm=False,
                 deg_cap=0, graph_seed=0, overdraw=1.25, threads=0) -> np.ndarray:
    """Return int32 [n_triples, 3] distinct (h, r, t) triples."""
    out = np.empty((n_triples, 3), dtype=np.int32)
    rc = _load().kgs_generate(n_entities, n_relations, n_triples, int(head_zipf), head_s,
                              int(tail_zipf), tail_s, int(rel_zipf), rel_s, int(shared_perm),
                              deg_cap, graph_seed, overdraw, out.ctypes.data, threads)
    if rc != n_triples:
        raise RuntimeError(f"kgs_generate failed with code {rc}")
    return out


def generate(cfg: "KGConfig | str", threads: int = 0) -> np.ndarray:
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    return generate_raw(cfg.n_entities, cfg.n_relations, cfg.n_triples,
                        head_zipf=cfg.head_zipf, head_s=cfg.head_s, tail_zipf=cfg.tail_zipf,
                        tail_s=cfg.tail_s, rel_zipf=cfg.rel_zipf, rel_s=cfg.rel_s,
                        shared_perm=cfg.shared_perm, deg_cap=cfg.deg_cap,
                        graph_seed=cfg.graph_seed, overdraw=cfg.extra.get("overdraw", 1.25),
                        threads=threads)


def random_tiny(rng: np.random.Generator, n_entities: int, n_relations: int, n_triples: int):
    """Small uniform triple sets (duplicates allowed) for oracle pins and parity edge cases."""
    h = rng.integers(0, n_entities, n_triples)
    r = rng.integers(0, n_relations, n_triples)
    t = rng.integers(0, n_entities, n_triples)
    return np.stack([h, r, t], axis=1).astype(np.int32)
