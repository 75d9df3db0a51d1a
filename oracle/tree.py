"""Tree-builder oracle: the budget-N candidate tree of highest plug-in score.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What the method computes (Sec. 3.2 Assumption 1, Sec. 3.3, Algorithm 1 second
step):

* One draft pass gives a marginal q_j over the vocabulary at every offset
  j = 1..L.  Here q_j = softmax(z_j) of the drafter's logits z_j, so
  log q_j(w) = z_j(w) - logsumexp(z_j)            (float64, ``log_marginals``).
* A string y_{1:l} (1 <= l <= L) has the plug-in score
  pi_hat(y) = prod_{j<=l} q_j(y_j); we rank by its logarithm, summed from the
  first offset on: s(y) = (...((log q_1(y_1)) + log q_2(y_2)) + ...).
* The tree keeps the N strings of highest score.  The kept set is prefix-closed
  because an extension never scores above its prefix (log q <= 0).

Readings where the paper is silent (each one is also listed in the design notes):

* Ties.  Exact score ties are common with bf16 logits (equal logits give equal
  terms), so the ranking needs a total order.  Tokens at offset j are ranked by
  (z_j desc, token index asc): r_j(w) is w's place in that order.  Strings are
  ordered by (score desc, length asc, (r_1, ..., r_l) lexicographic asc).  A
  prefix then always precedes its extensions and swapping a token for a
  better-ranked one never moves a string back, so the first N strings are
  prefix-closed and the children of every node carry the best-ranked tokens of
  their offset.
* Node numbering.  Node 0 is the root b; nodes 1..N are the kept strings in
  that order, so parents[i] < i.  parents[i] is the node of y_{1:l-1} (0 when
  l = 1) and tokens[i] = y_l.
* A row whose logits are all -inf has log q = -inf everywhere.  NaN and +inf
  logits are outside the contract.

Functions:

* ``log_marginals``       -- the definition of log q_j in float64;
* ``token_order``         -- each offset's tokens in rank order;
* ``ranked_strings_bruteforce`` -- every string of length 1..L scored and sorted
  (the definition written out; small vocabularies only);
* ``build_tree``          -- best-first enumeration of the same order, for full
  vocabularies: a max-heap that starts from the best 1-string and, when it
  emits a string, adds its best child (rank 0 at the next offset) and its next
  sibling (rank + 1 at the same offset).  Every string is reached from exactly
  one earlier string that precedes it in the order, so strings leave the heap
  in order;
* ``string_score``        -- s(y) of a given token string.
"""

import heapq
import itertools

import numpy as np


def _as_f64(z):
    if hasattr(z, "detach"):
        t = z.detach().to("cpu")
        if str(t.dtype) in ("torch.bfloat16", "torch.float16"):
            t = t.float()
        z = t.numpy()
    return np.asarray(z, dtype=np.float64)


def log_marginals(z):
    """log q_j(w) = z_j(w) - logsumexp_w z_j(w) for logits z [L][V] (Assumption 1)."""
    z = _as_f64(z)
    m = z.max(axis=-1, keepdims=True)
    out = np.full_like(z, -np.inf)
    finite = np.isfinite(m[..., 0])
    zf, mf = z[finite], m[finite]
    lse = mf + np.log(np.exp(zf - mf).sum(axis=-1, keepdims=True))
    out[finite] = zf - lse
    return out


def token_order(z):
    """order[j] = tokens of offset j sorted by (logit desc, index asc); rank[j][w] its inverse."""
    z = _as_f64(z)
    L, V = z.shape
    order = np.empty((L, V), dtype=np.int64)
    rank = np.empty((L, V), dtype=np.int64)
    for j in range(L):
        # np.lexsort sorts by the last key first: primary -z, secondary the index
        o = np.lexsort((np.arange(V), -z[j]))
        order[j] = o
        rank[j, o] = np.arange(V)
    return order, rank


def string_score(lq, toks):
    """s(y): the log plug-in score of token string ``toks``, summed from offset 1 on."""
    s = 0.0
    for j, t in enumerate(toks):
        s = s + float(lq[j, int(t)])
    return s


def ranked_strings_bruteforce(z, max_len=None):
    """Every string of length 1..L as (score, tokens), sorted by the total order.

    Exhaustive: V + V^2 + ... + V^L strings, so only for tiny inputs.
    """
    z = _as_f64(z)
    L, V = z.shape
    if max_len is not None:
        L = min(L, max_len)
    lq = log_marginals(z)
    _, rank = token_order(z)
    items = []
    for l in range(1, L + 1):
        for toks in itertools.product(range(V), repeat=l):
            s = string_score(lq, toks)
            key = (-s, l, tuple(int(rank[j, t]) for j, t in enumerate(toks)))
            items.append((key, s, toks))
    items.sort(key=lambda it: it[0])
    return [(s, toks) for _, s, toks in items]


def tree_from_strings(strings, root):
    """parents / tokens [N+1] of the tree whose node i (i >= 1) is strings[i-1]."""
    node_of = {(): 0}
    parents, tokens = [-1], [int(root)]
    for i, toks in enumerate(strings, start=1):
        toks = tuple(int(t) for t in toks)
        if toks[:-1] not in node_of:
            raise ValueError(f"string {toks} comes before its prefix")
        parents.append(node_of[toks[:-1]])
        tokens.append(toks[-1])
        node_of[toks] = i
    return np.asarray(parents, dtype=np.int64), np.asarray(tokens, dtype=np.int64)


def build_tree(z, root, budget):
    """The budget-N tree of Algorithm 1's second step for one sequence.

    z       draft logits [L][V] (offsets 1..L), any float dtype
    root    the pending root token b (node 0)
    budget  N, the number of kept strings

    Returns dict(parents, tokens, scores, strings): parents/tokens/scores have
    N + 1 entries (node 0 is the root, score 0), ``strings`` the token tuples
    of nodes 1..N.  Raises ValueError if fewer than N strings exist.
    """
    z = _as_f64(z)
    L, V = z.shape
    lq = log_marginals(z)
    order, _ = token_order(z)
    total = sum(V ** l for l in range(1, L + 1))
    if budget > total:
        raise ValueError(f"budget {budget} exceeds the {total} strings of length <= {L}")

    # heap entries: (key, prefix score, rank tuple); key = (-score, length, ranks)
    def entry(prefix_score, ranks):
        j = len(ranks) - 1
        s = prefix_score + float(lq[j, order[j, ranks[-1]]])
        return ((-s, len(ranks), ranks), prefix_score, s)

    heap = [entry(0.0, (0,))]
    strings, scores = [], [0.0]
    while len(strings) < budget:
        key, ps, s = heapq.heappop(heap)
        ranks = key[2]
        strings.append(tuple(int(order[j, r]) for j, r in enumerate(ranks)))
        scores.append(s)
        if len(ranks) < L:                       # best child: rank 0 at the next offset
            heapq.heappush(heap, entry(s, ranks + (0,)))
        if ranks[-1] + 1 < V:                    # next sibling: same prefix, next rank
            heapq.heappush(heap, entry(ps, ranks[:-1] + (ranks[-1] + 1,)))
    parents, tokens = tree_from_strings(strings, root)
    return {"parents": parents, "tokens": tokens, "scores": np.asarray(scores), "strings": strings}


def build_trees(logits, roots, budget):
    """``build_tree`` for every sequence of logits [batch][L][V]."""
    logits = _as_f64(logits)
    return [build_tree(logits[b], int(roots[b]), budget) for b in range(logits.shape[0])]
