"""Pins for the tree-builder oracle (CPU only): a hand-worked example, the
best-first enumeration against exhaustive enumeration, closed forms (one
offset, uniform rows, a dominant chain) and the structural invariants of the
kept set (prefix closure, nested budgets, sibling order)."""

import json
import math
import os

import numpy as np
import pytest

from oracle import tree as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_hand.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _hand_logits(g):
    return np.array([np.log(q) + c for q, c in zip(g["q"], g["offset_constant"])])


def test_hand_worked_example():
    g = _golden()
    z = _hand_logits(g)
    r = T.build_tree(z, g["root"], g["budget"])
    assert r["parents"].tolist() == g["parents"]
    assert r["tokens"].tolist() == g["tokens"]
    np.testing.assert_allclose(np.exp(r["scores"][1:]), g["products"][:g["budget"]], rtol=1e-12)
    full = T.build_tree(z, g["root"], len(g["order"]))
    assert [list(s) for s in full["strings"]] == g["order"]
    np.testing.assert_allclose(np.exp(full["scores"][1:]), g["products"], rtol=1e-12)
    bf = T.ranked_strings_bruteforce(z)
    assert [list(t) for _, t in bf] == g["order"]


def test_hand_example_needs_the_normaliser():
    # Without the per-offset log-normaliser the +3 / -2 constants would put
    # every 1-string ahead of every 2-string; the hand order interleaves them.
    g = _golden()
    r = T.build_tree(_hand_logits(g), g["root"], 3)
    assert [len(s) for s in r["strings"]] == [1, 2, 1]


def _random_logits(rng, L, V, kind):
    if kind == "normal":
        return rng.normal(0.0, 1.5, size=(L, V))
    if kind == "ties":                       # few distinct values: many exact ties
        return rng.integers(-2, 2, size=(L, V)).astype(float)
    if kind == "masked":
        z = rng.normal(0.0, 1.0, size=(L, V))
        z[rng.uniform(size=(L, V)) < 0.4] = -np.inf
        z[np.arange(L), rng.integers(0, V, size=L)] = 0.5   # at least one finite per row
        return z
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["normal", "ties", "masked"])
def test_best_first_equals_exhaustive_enumeration(kind):
    rng = np.random.default_rng(7)
    for L, V in [(1, 4), (2, 3), (3, 3), (4, 2), (2, 5), (3, 4)]:
        for _ in range(3):
            z = _random_logits(rng, L, V, kind)
            bf = T.ranked_strings_bruteforce(z)
            n_max = min(len(bf), 40)
            r = T.build_tree(z, 0, n_max)
            assert [tuple(s) for s in r["strings"]] == [t for _, t in bf[:n_max]], (L, V, kind)
            np.testing.assert_array_equal(r["scores"][1:], [s for s, _ in bf[:n_max]])
            for n in range(1, n_max):                # every smaller budget is a prefix
                rn = T.build_tree(z, 0, n)
                assert rn["strings"] == r["strings"][:n]


def test_one_offset_keeps_the_largest_logits():
    rng = np.random.default_rng(3)
    z = rng.integers(-5, 5, size=(1, 200)).astype(float)        # ties broken by lower index
    r = T.build_tree(z, 17, 63)
    want = np.argsort(-z[0], kind="stable")[:63]
    assert r["tokens"][1:].tolist() == want.tolist()
    assert r["parents"].tolist() == [-1] + [0] * 63


def test_uniform_rows_closed_form():
    V, L = 3, 3
    z = np.zeros((L, V))
    r = T.build_tree(z, 0, V + V * V + 5)
    # every string of length l scores -l log V: all 1-strings, then 2-strings in
    # lexicographic token order, then 3-strings
    strings = r["strings"]
    assert strings[:V] == [(t,) for t in range(V)]
    assert strings[V:V + V * V] == [(a, b) for a in range(V) for b in range(V)]
    assert strings[V + V * V:] == [(0, 0, t) for t in range(3)] + [(0, 1, 0), (0, 1, 1)]
    lens = np.array([len(s) for s in strings])
    np.testing.assert_allclose(r["scores"][1:], -lens * math.log(V), rtol=1e-14)


def test_dominant_token_per_offset_gives_a_chain_first():
    V, L = 100, 7
    rng = np.random.default_rng(5)
    dom = rng.choice(V, size=L, replace=False)
    z = np.zeros((L, V))
    z[np.arange(L), dom] = 40.0                  # q(dominant) = 1 - 99 e^-40
    r = T.build_tree(z, 1, L + 3)
    assert r["parents"][:L + 1].tolist() == list(range(-1, L))
    assert r["tokens"][1:L + 1].tolist() == dom.tolist()
    # every string with one non-dominant token then scores -40 (in float64 the
    # dominant terms round to 0), and the shortest of them wins the tie: the
    # runner-up of the first offset, the lowest non-dominant index
    runner = 0 if dom[0] != 0 else 1
    assert r["strings"][L] == (runner,)


def test_all_minus_inf_row_scores_minus_inf():
    z = np.array([[0.0, 1.0, -np.inf], [-np.inf, -np.inf, -np.inf]])
    lq = T.log_marginals(z)
    assert np.all(np.isneginf(lq[1]))
    r = T.build_tree(z, 0, 4)
    assert r["strings"][:2] == [(1,), (0,)]
    assert np.isneginf(r["scores"][3]) and np.isneginf(r["scores"][4])


def test_structure_on_draft_like_rows():
    rng = np.random.default_rng(11)
    L, V = 10, 500
    z = rng.normal(0, 1, size=(L, V))
    for j in range(L):
        z[j, rng.choice(V, 3, replace=False)] = [9 - 0.5 * j, 8 - 0.5 * j, 7 - 0.5 * j]
    r = T.build_tree(z, 3, 63)
    par, strings, lq = r["parents"], r["strings"], T.log_marginals(z)
    order, rank = T.token_order(z)
    node_of = {s: i + 1 for i, s in enumerate(strings)}
    for i, s in enumerate(strings, start=1):
        assert 0 <= par[i] < i
        assert len(s) <= L
        assert (s[:-1] == () and par[i] == 0) or node_of[s[:-1]] == par[i]
        rk = rank[len(s) - 1, s[-1]]
        if rk > 0:                            # previous sibling kept and earlier
            prev = s[:-1] + (int(order[len(s) - 1, rk - 1]),)
            assert node_of[prev] < i
        assert r["scores"][i] == T.string_score(lq, s)
    assert np.all(np.diff(r["scores"][1:]) <= 0)
    assert max(len(s) for s in strings) >= 4


def test_budget_beyond_the_string_count_raises():
    with pytest.raises(ValueError):
        T.build_tree(np.zeros((2, 2)), 0, 7)      # 2 + 4 strings
    assert len(T.build_tree(np.zeros((2, 2)), 0, 6)["strings"]) == 6
