"""Parity of membership verification (smore_verify) with the CPU oracle,
bit for bit, and the evaluation workflow on nested graphs it serves
(appendix on the task setup): queries sampled on G_test, their positives
verified against G_valid and G_train to find the answers missing there,
and filtered negatives of G_test for every query."""
import numpy as np
import pytest

import kgsynth
import paper_2110_14890_amd as sm
from gpu_common import assert_same, config_graph, gpu_sample, graph_pair, progress, require_gpu

pytestmark = pytest.mark.gpu


def gpu_verify(g, qt, anchors, relations, cand):
    import torch
    dev = torch.device("cuda")
    out = sm.verify(g, qt, torch.as_tensor(anchors, device=dev), torch.as_tensor(relations, device=dev),
                    torch.as_tensor(cand, device=dev))
    torch.cuda.synchronize()
    return out["mask"].cpu().numpy().view(np.uint32), out["n_valid"].cpu().numpy()


@pytest.mark.parametrize("qt", sm.TYPES)
def test_verify_parity_random_candidates(qt):
    require_gpu()
    rng = np.random.default_rng(31)
    tr = kgsynth.random_tiny(rng, 3000, 6, 60000)
    g, og = graph_pair(tr, 3000, 6, True)
    q = og.sample(qt, 300, 0, seed=1, neg_tries=0)
    anchors, relations = q["anchors"].copy(), q["relations"].copy()
    anchors[7] = 5000            # out of range: the query is refused, its row is zero
    for n in (37, 600):
        progress(f"verify {qt} n {n}")
        cand = rng.integers(-3, 3003, size=(300, n)).astype(np.int32)
        cand[:, 0] = q["positive"]  # the positive answers its own query
        mask, nv = gpu_verify(g, qt, anchors, relations, cand)
        ref = og.verify(qt, anchors, relations, cand)
        assert np.array_equal(mask, ref["mask"]) and np.array_equal(nv, ref["n_valid"]), f"{qt} n {n}"
        assert nv[7] == -1


def test_evaluation_on_nested_graphs():
    """G_train within G_valid within G_test (90 / 5 / 5 % of the triples):
    test queries with 1,000 filtered negatives from G_test; their positives
    verified on G_valid and G_train; everything against the oracle."""
    require_gpu()
    cfg, tr = config_graph("fb15k237")
    perm = np.random.default_rng(7).permutation(len(tr))
    n_tr, n_va = int(0.9 * len(tr)), int(0.95 * len(tr))
    parts = {"train": tr[perm[:n_tr]], "valid": tr[perm[:n_va]], "test": tr}
    graphs = {k: graph_pair(v, cfg.n_entities, cfg.n_relations) for k, v in parts.items()}
    for qt in ("1p", "2p", "3p", "2i", "ip", "pi"):
        progress(f"evaluation {qt}")
        g, og = graphs["test"]
        got = gpu_sample(g, qt, 512, 1000, seed=11, neg_tries=4000)
        ref = og.sample(qt, 512, 1000, seed=11, neg_tries=4000)
        assert_same(got, ref, what=f"test-graph negatives {qt}")
        pos = got["positive"][:, None].copy()
        hard = {}
        for part in ("valid", "train"):
            gp, ogp = graphs[part]
            mask, nv = gpu_verify(gp, qt, got["anchors"], got["relations"], pos)
            r = ogp.verify(qt, got["anchors"], got["relations"], pos)
            assert np.array_equal(mask, r["mask"]) and np.array_equal(nv, r["n_valid"]), part
            hard[part] = (mask[:, 0] & 1).astype(bool)
        ok = got["n_valid"] >= 0
        # answers missing from G_valid are missing from G_train too
        assert (hard["train"][ok] >= hard["valid"][ok]).all()
        assert hard["train"][ok].any()


def test_verify_and_sample_without_candidates():
    """n = 0 candidates per query: smore_verify writes only n_valid (0, or
    -1 for a query with an out-of-range anchor), and smore_sample with
    n_neg = 0 writes n_valid and neg_draws = 0 (or -1 without a positive);
    neither needs a workspace (the binding passes NULL)."""
    require_gpu()
    rng = np.random.default_rng(41)
    tr = kgsynth.random_tiny(rng, 500, 4, 6000)
    g, og = graph_pair(tr, 500, 4, True)
    for qt in sm.TYPES:
        progress(f"no candidates {qt}")
        q = og.sample(qt, 64, 0, seed=2, neg_tries=0)
        anchors, relations = q["anchors"].copy(), q["relations"].copy()
        anchors[3] = 900
        mask, nv = gpu_verify(g, qt, anchors, relations, np.zeros((64, 0), np.int32))
        ref = og.verify(qt, anchors, relations, np.zeros((64, 0), np.int32))
        assert mask.size == 0 and np.array_equal(nv, ref["n_valid"]), qt
        got = gpu_sample(g, qt, 64, 0, seed=2, neg_tries=0)
        assert_same(got, og.sample(qt, 64, 0, seed=2, neg_tries=0), what=f"{qt} n_neg 0")
