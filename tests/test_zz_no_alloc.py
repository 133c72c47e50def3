"""The entry point that allocates nothing (smore_sample_noalloc): its rows
equal smore_sample's, element by element (integer work, tolerance 0), on two
calls in a row, the second with a smaller input, so that the fixed scratch
still holding the first call's contents cannot change a result; and
arguments that need more scratch than the fixed size are refused."""
import numpy as np
import pytest

import kgsynth
import paper_2110_14890_amd as sm
from gpu_common import FIELDS, graph_pair, progress, require_gpu, to_numpy

pytestmark = pytest.mark.gpu


def _both(g, qt, batch, n_neg, neg_tries, seed, query_offset):
    dag = sm.query_preset(qt)
    args = sm.make_args(batch, n_neg, seed=seed, query_offset=query_offset, neg_tries=neg_tries)
    fixed = sm.alloc_outputs(batch, n_neg)
    for v in fixed.values():
        v.fill_(-7)
    sm.sample_noalloc_into(g, dag, args, fixed)
    ref = sm.sample_into(g, dag, args, sm.alloc_outputs(batch, n_neg))
    return to_numpy(fixed), to_numpy(ref)


def test_noalloc_equals_smore_sample_on_consecutive_calls():
    require_gpu()
    rng = np.random.default_rng(5)
    tr = kgsynth.random_tiny(rng, 4000, 7, 90000)
    g, _ = graph_pair(tr, 4000, 7, True)
    # (batch, n_neg, neg_tries): a large call, then a smaller one over the
    # same scratch, then one with more draw rounds per query
    for qt in ("3p", "ip", "pi", "2u", "pni"):
        for batch, n_neg, tries, off in ((1500, 200, 800, 0), (300, 37, 90, 7), (64, 5, 4096, 99)):
            progress(f"noalloc {qt} batch {batch} n_neg {n_neg} tries {tries}")
            got, ref = _both(g, qt, batch, n_neg, tries, seed=3, query_offset=off)
            for k in FIELDS:
                assert np.array_equal(got[k], ref[k]), (qt, batch, k)
            assert (ref["n_valid"] >= 0).any()


def test_noalloc_refuses_more_than_its_scratch():
    require_gpu()
    rng = np.random.default_rng(6)
    tr = kgsynth.random_tiny(rng, 100, 2, 800)
    g, _ = graph_pair(tr, 100, 2, False)
    dag = sm.query_preset("2p")
    big = sm.make_args(16384, 512, neg_tries=2048)
    assert sm.workspace_bytes(dag, big) > sm.NOALLOC_SCRATCH_BYTES
    with pytest.raises(sm.SmoreError) as e:
        sm.sample_noalloc_into(g, dag, big, sm.alloc_outputs(16384, 512))
    assert e.value.code == -3 and "scratch" in str(e.value)
    # the same call without negatives needs no scratch at all
    out = sm.sample_noalloc_into(g, dag, sm.make_args(16384, 0), sm.alloc_outputs(16384, 0))
    ref = sm.sample(g, "2p", 16384, 0)
    got = to_numpy(out)
    ref = to_numpy(ref)
    for k in FIELDS:
        assert np.array_equal(got[k], ref[k]), k
