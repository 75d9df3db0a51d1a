"""Greedy acceptance oracle: per-row vocabulary argmax and the walk of Algorithm 1.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

* ``argmax_rows``  -- t_v = argmax_w rows[v](w), the target-greedy token of every
  verified row (Algorithm 1, App. B).  Ties go to the lowest index, as numpy's
  argmax does (it returns the first maximum); a NaN counts as larger than every
  number and the first NaN wins, again numpy's rule.  +0 and -0 compare equal.
* ``accepted_length_def1`` -- Def. 1 (Sec. 3.3) evaluated directly, the
  oracle's definition of acceptance: A(T) = max{k >= 0 : Y_{1:j} in T for all
  j <= k}, the depth of the deepest node whose every edge carries the argmax
  token of its parent's row.  For every node it climbs to the root and checks
  the edges.  In a tree of distinct strings (distinct tokens among siblings)
  that node is unique; the accepted path is its root chain and the bonus
  token is its own row's argmax.
* ``greedy_walk``  -- the same acceptance reached by descending from the root
  (the form Algorithm 1 takes), kept as a cross-check: from each node, the
  child whose edge token equals the node's argmax, if there is one.  A
  malformed tree may give two siblings one token; the descent then takes the
  lower index (the reading the library documents), where Def. 1's deepest
  node need not be unique, so ``greedy_accept`` uses the descent for such
  trees (and for parents arrays that are no tree).  Only children after their parent count (every child in a tree), so
  the descent ends within n steps whatever the parents array holds.

* ``row_entropy``  -- H = -sum_w p(w) log p(w) of p = softmax(row), in nats: the
  target's next-token entropy, which the paper's entropy law (Sec. 4) reads at
  the round root (row 0).  -inf logits carry probability 0.

A round commits a + 1 tokens: the a accepted tree tokens and the bonus token
read off the last verified row (Sec. 3.1, Eq. 1).
"""

import numpy as np


def argmax_rows(logits):
    """Row-wise argmax with lowest-index ties; logits [..., V] of any float dtype."""
    if hasattr(logits, "detach"):
        t = logits.detach().to("cpu")
        if str(t.dtype) in ("torch.bfloat16", "torch.float16"):
            t = t.float()
        logits = t.numpy()
    x = np.asarray(logits, dtype=np.float64)
    return np.argmax(x, axis=-1).astype(np.int64)


def greedy_walk(argmax_row, parents, tokens):
    """Acceptance by descent over one packed tree (cross-check of Def. 1).

    argmax_row [n]  target-greedy token of each node's row
    parents    [n]  parents[0] = -1
    tokens     [n]  tokens[0] = root b; tokens[c] is the token on the edge into c

    Returns (a, path, next_root): a accepted non-root tokens, path = node ids
    from the root to the last accepted node (length a + 1), and next_root =
    argmax_row[path[-1]], the bonus token that becomes the next root.
    """
    parents = [int(p) for p in parents]
    tokens = [int(t) for t in tokens]
    argmax_row = [int(t) for t in argmax_row]
    path = [0]
    while True:
        v = path[-1]
        # children of v after v carrying v's argmax token, lowest index first
        # (in a tree every child comes after its parent, so this is every child)
        match = [c for c in range(v + 1, len(parents)) if parents[c] == v and tokens[c] == argmax_row[v]]
        if not match:
            return len(path) - 1, path, argmax_row[v]
        path.append(match[0])


def accepted_length_def1(argmax_row, parents, tokens):
    """Def. 1 evaluated directly: the deepest node whose whole root path is target-greedy.

    Returns (a, path) where path is that node's chain from the root (the root
    alone when no child of the root matches).
    """
    parents = [int(p) for p in parents]
    tokens = [int(t) for t in tokens]
    argmax_row = [int(t) for t in argmax_row]
    best_depth, best_node = 0, 0
    for c in range(len(parents)):
        chain = [c]
        while parents[chain[-1]] >= 0:
            chain.append(parents[chain[-1]])
        chain.reverse()  # root ... c
        ok = all(tokens[chain[k + 1]] == argmax_row[chain[k]] for k in range(len(chain) - 1))
        depth = len(chain) - 1
        if ok and depth > best_depth:
            best_depth, best_node = depth, c
    path = [best_node]
    while parents[path[-1]] >= 0:
        path.append(parents[path[-1]])
    path.reverse()
    return best_depth, path


def _tree_of_strings(parents, tokens):
    """parents[0] = -1, every parent before its child, distinct tokens among
    siblings: the packed tree is a set of distinct strings (Def. 1)."""
    if int(parents[0]) != -1:
        return False
    seen = set()
    for c in range(1, len(parents)):
        key = (int(parents[c]), int(tokens[c]))
        if not 0 <= key[0] < c or key in seen:
            return False
        seen.add(key)
    return True


def greedy_accept(logits, parents, tokens, path_stride=None):
    """Batched acceptance: argmax of every row, then each sequence's accepted
    path by Def. 1 (by descent where the parents and tokens do not form a tree
    of distinct strings).

    logits [batch][n][V]; parents, tokens [batch][n].
    Returns dict with argmax [batch][n], accept_len [batch], accept_path
    [batch][path_stride] (-1 padded), next_root [batch], committed (list of the
    a + 1 committed tokens per sequence).
    """
    am = argmax_rows(logits)
    parents = np.asarray(parents if not hasattr(parents, "numpy") else parents.cpu().numpy())
    tokens = np.asarray(tokens if not hasattr(tokens, "numpy") else tokens.cpu().numpy())
    batch, n = am.shape
    if path_stride is None:
        path_stride = n
    acc = np.zeros(batch, dtype=np.int64)
    paths = -np.ones((batch, path_stride), dtype=np.int64)
    roots = np.zeros(batch, dtype=np.int64)
    committed = []
    for b in range(batch):
        if _tree_of_strings(parents[b], tokens[b]):
            a, path = accepted_length_def1(am[b], parents[b], tokens[b])
            nr = int(am[b][path[-1]])
            assert (a, path, nr) == greedy_walk(am[b], parents[b], tokens[b])
        else:
            a, path, nr = greedy_walk(am[b], parents[b], tokens[b])
        acc[b] = a
        k = min(len(path), path_stride)
        paths[b, :k] = path[:k]
        roots[b] = nr
        committed.append([int(tokens[b][c]) for c in path[1:]] + [int(nr)])
    return {"argmax": am, "accept_len": acc, "accept_path": paths, "next_root": roots,
            "committed": committed}


def row_entropy(row):
    """Entropy in nats of softmax(row) for one row of logits (float64)."""
    if hasattr(row, "detach"):
        t = row.detach().to("cpu")
        if str(t.dtype) in ("torch.bfloat16", "torch.float16"):
            t = t.float()
        row = t.numpy()
    z = np.asarray(row, dtype=np.float64)
    z = z[np.isfinite(z)]
    m = z.max()
    e = np.exp(z - m)
    s = e.sum()
    p = e / s
    return float(-(p * ((z - m) - np.log(s))).sum())
