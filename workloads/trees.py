"""Seeded candidate-tree generators (inputs only: no step of the method is computed here).

A candidate tree (Def. 1) is stored as two int32 arrays of length n:
``parents`` (parents[0] = -1 for the root b, 0 <= parents[i] < i) and
``tokens`` (tokens[0] = b, tokens[c] = the token on the edge into c, distinct
among siblings because the tree is a set of strings).

``best_first_tree`` mimics the shape of the paper's top-N-by-plug-in-score trees
(Sec. 3.3): it repeatedly expands the highest-scoring frontier node, so trees
have a deep high-probability spine with bushy side branches.
"""

import numpy as np


def _rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def best_first_tree(n, depth_cap, branch_choices, vocab, key):
    """Grow an n-node tree (root included) best-first.

    The root has score 1.  Repeatedly the highest-score unexpanded node whose
    depth is below ``depth_cap`` (ties: lowest index) gets k children, k drawn
    from ``branch_choices``; child rank r gets score parent * c * 2**-r with
    c ~ U(0.5, 0.95).  If every node below the cap is already expanded, the
    best one gets one more child.  Nodes are numbered in creation order.
    """
    rng = _rng(*key)
    parents, depth, score, expanded, nkids = [-1], [0], [1.0], [False], [0]
    if n > 1 and depth_cap < 1:
        raise ValueError("depth cap too small for the requested node count")
    while len(parents) < n:
        frontier = [i for i in range(len(parents)) if not expanded[i] and depth[i] < depth_cap]
        if frontier:
            v = max(frontier, key=lambda i: (score[i], -i))
            expanded[v] = True
            k = int(rng.choice(branch_choices))
        else:  # every node below the cap is expanded: widen the best one by one more child
            v = max((i for i in range(len(parents)) if depth[i] < depth_cap), key=lambda i: (score[i], -i))
            k = 1
        for _ in range(k):
            if len(parents) == n:
                break
            c = rng.uniform(0.5, 0.95)
            parents.append(v)
            depth.append(depth[v] + 1)
            score.append(score[v] * c * 2.0 ** (-nkids[v]))
            expanded.append(False)
            nkids.append(0)
            nkids[v] += 1
    tokens = assign_tokens(parents, vocab, rng)
    return np.asarray(parents, dtype=np.int32), tokens


def assign_tokens(parents, vocab, rng):
    """Uniform tokens, distinct among the children of each node; the root token is uniform."""
    n = len(parents)
    tokens = np.zeros(n, dtype=np.int32)
    tokens[0] = rng.integers(0, vocab)
    kids = {}
    for c in range(1, n):
        kids.setdefault(int(parents[c]), []).append(c)
    for p, cs in kids.items():
        if len(cs) > vocab:
            raise ValueError("more siblings than vocabulary entries")
        toks = rng.choice(vocab, size=len(cs), replace=False)
        for c, t in zip(cs, toks):
            tokens[c] = int(t)
    return tokens


def chain_tree(n, vocab, key):
    """A chain: parents[i] = i - 1 (a linear draft of n - 1 tokens after the root)."""
    rng = _rng(*key)
    parents = np.arange(-1, n - 1, dtype=np.int32)
    return parents, assign_tokens(parents, vocab, rng)


def star_tree(n, vocab, key):
    """A star: every non-root node is a child of the root (depth 1)."""
    rng = _rng(*key)
    parents = np.zeros(n, dtype=np.int32)
    parents[0] = -1
    return parents, assign_tokens(parents, vocab, rng)


def node_depths(parents):
    d = np.zeros(len(parents), dtype=np.int64)
    for i in range(1, len(parents)):
        d[i] = d[parents[i]] + 1
    return d
