"""Brute-force node cuts and their cost (test infrastructure only).

Node cut (Sec. 3.2, Def. "Node cut"): a set of plan nodes meeting every
anchor-to-root path exactly once.  Cost of a cut for one path of t
projections whose cut node lies after i of them: max(C^i, C^(t-i)); the
optimal-scheduling objective minimises, over cuts, the maximum of that cost
over the anchors.  Costs are kept as exponents of C (the appendix on the DP
measures cost on a logarithmic scale).

A plan is given as (op, child, root): op[k] in {0 anchor, 1 projection,
2 and, 3 or}; child[k] lists up to three children (-1 unused).
"""
from itertools import combinations


def parents(op, child):
    par = [-1] * len(op)
    for k in range(len(op)):
        for c in child[k]:
            if c >= 0:
                par[c] = k
    return par


def anchor_paths(op, child, root):
    """For each anchor, its path [anchor, ..., root] as node ids."""
    par = parents(op, child)
    paths = []
    for k in range(len(op)):
        if op[k] == 0:
            p = [k]
            while p[-1] != root:
                p.append(par[p[-1]])
            paths.append(p)
    return paths


def is_cut(op, child, root, cut):
    return all(sum(1 for v in p if v in cut) == 1 for p in anchor_paths(op, child, root))


def cost(op, child, root, cut):
    """max over anchor paths of max(i, t - i) (exponent of C)."""
    worst = 0
    for p in anchor_paths(op, child, root):
        proj = [1 if op[p[m + 1]] == 1 else 0 for m in range(len(p) - 1)]  # edge p[m] -> p[m+1]
        t = sum(proj)
        pos = next(m for m, v in enumerate(p) if v in cut)
        i = sum(proj[:pos])
        worst = max(worst, i, t - i)
    return worst


def all_cuts(op, child, root):
    n = len(op)
    out = []
    for size in range(1, n + 1):
        for cut in combinations(range(n), size):
            if is_cut(op, child, root, set(cut)):
                out.append(frozenset(cut))
    return out


def optimal(op, child, root):
    """(minimum cost, list of cuts achieving it)."""
    cuts = all_cuts(op, child, root)
    best = min(cost(op, child, root, c) for c in cuts)
    return best, [c for c in cuts if cost(op, child, root, c) == best]


def mask(cut):
    m = 0
    for v in cut:
        m |= 1 << v
    return m


def strict(op, child, root):
    """The optimal cut the DP's top-down construction returns with a strict
    comparison (appendix on the optimal cut: a node joins the cut only when
    its children's best cost is larger): among the optimal cuts, the one
    that caches least far forward, i.e. with the smallest total number of
    projections between the anchors and their cut node."""
    best, cand = optimal(op, child, root)

    def forward_depth(cut):
        total = 0
        for p in anchor_paths(op, child, root):
            pos = next(m for m, v in enumerate(p) if v in cut)
            total += sum(1 for m in range(pos) if op[p[m + 1]] == 1)
        return total

    return min(cand, key=lambda c: (forward_depth(c), sorted(c)))
