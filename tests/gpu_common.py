"""Helpers shared by the GPU tests: run the HIP path and the oracle on the
same seeded inputs and compare every output array element by element."""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import kgsynth
import oracle
import paper_2110_14890_amd as sm

FIELDS = sm.OUT_FIELDS


def progress(msg: str) -> None:
    """Progress line that bypasses pytest's capture (long GPU tests)."""
    print(f"[gpu-test] {msg}", file=sys.__stderr__, flush=True)


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    if not __import__("os").path.exists(sm.LIB_PATH):
        pytest.fail("libsmore.so is not built")


def to_numpy(out: dict) -> dict:
    import torch
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def gpu_sample(g, qtype, batch, n_neg, **kw) -> dict:
    return to_numpy(sm.sample(g, qtype, batch, n_neg, **kw))


def assert_same(gpu: dict, ref: dict, rows=None, what=""):
    for k in FIELDS:
        a = gpu[k] if rows is None else gpu[k][rows]
        b = ref[k]
        if not np.array_equal(a, b):
            bad = np.nonzero((a != b).reshape(len(a), -1).any(axis=1))[0]
            i = int(bad[0])
            raise AssertionError(f"{what} field {k}: {len(bad)} rows differ; first row {i}: "
                                 f"gpu {a[i]} vs oracle {b[i]}")


def oracle_rows(og, qtype, qids, n_neg, seed, neg_tries, pos_tries=64, max_fanout=0, threads=16):
    """Oracle outputs for an arbitrary list of query ids (one call per id, in
    parallel; the oracle's per-call loop releases the GIL)."""
    def one(q):
        return og.sample(qtype, 1, n_neg, seed=seed, query_offset=int(q), pos_tries=pos_tries,
                         neg_tries=neg_tries, max_fanout=max_fanout, threads=1)
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(one, qids))
    return {k: np.concatenate([r[k] for r in res]) for k in FIELDS}


def graph_pair(triples, V, R, add_inverse=False):
    return (sm.Graph(triples, V, R, add_inverse), oracle.Graph(triples, V, R, add_inverse))


def config_graph(name):
    cfg = kgsynth.CONFIGS[name]
    tr = kgsynth.generate(cfg)
    return cfg, tr
