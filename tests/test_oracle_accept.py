"""Pins for the acceptance oracle (CPU only): argmax semantics, Algorithm 1's walk
against Def. 1 evaluated directly, exhaustive small trees, and hand-worked cases."""

import itertools

import numpy as np
import pytest
import torch

from oracle import accept as C


# ---------------------------------------------------------------- argmax
def test_argmax_unique_and_lowest_index_ties():
    row = np.array([0.5, 3.0, -1.0, 3.0, 2.9])
    assert C.argmax_rows(row[None])[0] == 1               # tie at 1 and 3 -> 1
    row = np.full(11, -2.0)
    row[0] = row[10] = 7.0
    assert C.argmax_rows(row[None])[0] == 0               # first and last -> first
    row = np.arange(9, dtype=float)
    assert C.argmax_rows(row[None])[0] == 8


def test_argmax_signed_zero_ties_and_nan():
    row = np.full(8, -1.0)
    row[5], row[3] = -0.0, 0.0
    assert C.argmax_rows(row[None])[0] == 3
    row[5], row[3] = 0.0, -0.0
    assert C.argmax_rows(row[None])[0] == 3               # -0 == +0: lowest index still wins
    row = np.array([1.0, np.nan, 5.0, np.nan])
    assert C.argmax_rows(row[None])[0] == 1               # first NaN wins


def test_argmax_bf16_rows():
    t = torch.tensor([[1.0, 2.0, 2.0, -3.0]], dtype=torch.bfloat16)
    assert C.argmax_rows(t)[0] == 1


# ---------------------------------------------------------------- walk
def test_hand_worked_walk():
    # root 0 (token 10): children 1 (5), 2 (6); node 1: children 3 (7), 4 (8);
    # node 2: child 5 (9); node 4: child 6 (3).
    parents = [-1, 0, 0, 1, 1, 2, 4]
    tokens = [10, 5, 6, 7, 8, 9, 3]
    argmax = [5, 8, 0, 0, 3, 0, 42]   # 0 -> 1 -> 4 -> 6, then 42 is no child of 6
    a, path, nr = C.greedy_walk(argmax, parents, tokens)
    assert (a, path, nr) == (3, [0, 1, 4, 6], 42)
    res = C.greedy_accept(np.eye(64)[argmax][None], [parents], [tokens])
    assert res["committed"][0] == [5, 8, 3, 42]           # a + 1 tokens (Eq. 1)


def test_root_mismatch_commits_only_the_bonus_token():
    parents, tokens = [-1, 0, 0], [1, 2, 3]
    a, path, nr = C.greedy_walk([99, 2, 3], parents, tokens)
    assert (a, path, nr) == (0, [0], 99)


def test_chain_fully_planted_accepts_whole_chain():
    n = 16
    parents = list(range(-1, n - 1))
    tokens = [100 + i for i in range(n)]
    argmax = [tokens[i + 1] for i in range(n - 1)] + [7]
    a, path, nr = C.greedy_walk(argmax, parents, tokens)
    assert a == n - 1 and path == list(range(n)) and nr == 7


def _increasing_trees(n):
    for choice in itertools.product(*[range(i) for i in range(1, n)]):
        yield [-1] + list(choice)


def test_walk_equals_def1_exhaustively_on_small_trees():
    """All increasing trees with up to 6 nodes; children labelled 0,1,2,... in index order
    (distinct siblings); every argmax assignment over the alphabet {0,1,2}."""
    checked = 0
    for n in range(1, 7):
        for parents in _increasing_trees(n):
            tokens = [0] * n
            seen = {}
            for c in range(1, n):
                tokens[c] = seen.get(parents[c], 0)
                seen[parents[c]] = tokens[c] + 1
            depth = [0] * n
            for c in range(1, n):
                depth[c] = depth[parents[c]] + 1
            for am in itertools.product(range(3), repeat=n):
                a, path, nr = C.greedy_walk(am, parents, tokens)
                a2, path2 = C.accepted_length_def1(am, parents, tokens)
                assert (a, path) == (a2, path2)
                assert a <= max(depth)
                for k in range(a):                      # every committed token is a parent-row argmax
                    assert tokens[path[k + 1]] == am[path[k]]
                last = path[-1]
                assert nr == am[last]
                assert nr not in [tokens[c] for c in range(n) if parents[c] == last]
                checked += 1
    assert checked > 80000


def test_duplicate_sibling_tokens_take_lowest_index_child():
    parents, tokens = [-1, 0, 0, 2], [0, 4, 4, 9]
    a, path, nr = C.greedy_walk([4, 1, 9, 5], parents, tokens)
    assert path == [0, 1] and nr == 1


def test_batched_accept_padding_and_outputs():
    parents = np.array([[-1, 0, 1, 1], [-1, 0, 0, 0]])
    tokens = np.array([[0, 5, 6, 7], [0, 1, 2, 3]])
    logits = np.zeros((2, 4, 10))
    logits[0, 0, 5] = logits[0, 1, 7] = logits[0, 3, 2] = 1.0   # 0->1->3, bonus 2
    logits[1, 0, 9] = 1.0                                         # no match at the root
    res = C.greedy_accept(logits, parents, tokens, path_stride=5)
    assert res["accept_len"].tolist() == [2, 0]
    assert res["accept_path"].tolist() == [[0, 1, 3, -1, -1], [0, -1, -1, -1, -1]]
    assert res["next_root"].tolist() == [2, 9]
    assert res["argmax"].tolist() == [[5, 7, 0, 2], [9, 0, 0, 0]]


# ---------------------------------------------------------------- root entropy
def test_entropy_closed_forms():
    assert abs(C.row_entropy(np.zeros(1000)) - np.log(1000)) < 1e-12          # uniform: log V
    row = np.full(50, -np.inf)
    row[[3, 40]] = 7.0
    assert abs(C.row_entropy(row) - np.log(2)) < 1e-12                         # two equal masses
    row = np.log(np.array([0.5, 0.25, 0.25])) + 3.0
    assert abs(C.row_entropy(row) - 1.5 * np.log(2)) < 1e-12                   # p = 1/2, 1/4, 1/4
    row = np.array([0.0, -1e4, -1e4])
    assert C.row_entropy(row) < 1e-300 + 1e-12                                 # nearly one-hot


def test_entropy_is_shift_invariant_and_bounded():
    rng = np.random.default_rng(2)
    row = rng.normal(0, 2, size=5000)
    h = C.row_entropy(row)
    assert abs(C.row_entropy(row + 123.0) - h) < 1e-9
    assert 0.0 < h < np.log(5000)
