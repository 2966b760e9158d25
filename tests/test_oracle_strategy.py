"""Pins of the strategy-selection oracle (oracle.strategy), CPU only.

* the selected sets are, for every n, the heaviest connected subtrees of n
  nodes containing the root (brute force over all subtrees of small trees);
* with an exact (bucket-free) cost that grows linearly in the tree size, the
  objective is unimodal and the early-stopping search returns the global
  argmax (the sugar-water inequality of Section 5.3);
* the cost formula and the bucket rule on hand-computed values;
* the least-squares fit recovers known coefficients from exact data;
* plausible mistakes planted in copies of the oracle fail these checks.
"""

import itertools
import math

import numpy as np
import pytest

from oracle import strategy as S


def random_tree(rng, n, max_children=3):
    parents, kids = [-1], [0]
    for i in range(1, n):
        cands = [j for j in range(i) if kids[j] < max_children]
        p = int(rng.choice(cands))
        parents.append(p)
        kids[p] += 1
        kids.append(0)
    return parents


def monotone_weights(rng, parents):
    """w(root) = 1, w(child) = w(parent) * o with sibling o's summing to <= 1
    (draft logits times a linear F)."""
    w = [1.0]
    for i in range(1, len(parents)):
        w.append(w[parents[i]] * float(rng.uniform(0.05, 0.6)))
    return w


def connected_subsets(parents, n):
    """Every node set of size n that contains the root and each member's parent."""
    nodes = range(1, len(parents))
    for comb in itertools.combinations(nodes, n - 1):
        s = set(comb) | {0}
        if all(parents[i] in s for i in comb):
            yield s


@pytest.mark.parametrize("seed", range(12))
def test_selected_sets_are_heaviest_connected_subtrees(seed):
    rng = np.random.default_rng(seed)
    parents = random_tree(rng, int(rng.integers(2, 10)))
    w = monotone_weights(rng, parents)
    order = S.selection_order(parents, w)
    for n in range(1, len(parents) + 1):
        chosen = set(order[:n])
        assert all(parents[i] in chosen for i in chosen if i), "prefix not connected"
        best = max(sum(w[i] for i in s) for s in connected_subsets(parents, n))
        assert math.isclose(sum(w[i] for i in chosen), best, rel_tol=1e-12)


def test_ties_go_to_the_shallower_then_lower_index():
    parents = [-1, 0, 0, 1, 2]
    w = [1.0, 0.5, 0.5, 0.5, 0.25]
    assert S.selection_order(parents, w) == [0, 1, 2, 3, 4]
    parents = [-1, 0, 1, 0]
    w = [1.0, 0.5, 0.5, 0.5]
    assert S.selection_order(parents, w) == [0, 1, 3, 2]


@pytest.mark.parametrize("seed", range(8))
def test_early_stopping_finds_the_argmax_when_unimodal(seed):
    """Every tree has at least n_max nodes, so each step adds one node per
    sample: the time increment is constant while the accepted-length
    increment (sorted weights) never grows, the premise of the sugar-water
    argument.  (When a small tree runs out, the time increment shrinks and
    the objective can rise again; the search then still returns the best
    objective it saw.)"""
    rng = np.random.default_rng(100 + seed)
    trees = []
    for _ in range(int(rng.integers(1, 5))):
        p = random_tree(rng, int(rng.integers(48, 80)))
        trees.append((p, monotone_weights(rng, p)))
    lens = [int(x) for x in rng.integers(100, 5000, len(trees))]
    coeffs = {"c0": float(rng.uniform(1, 10)), "c_seq": 1e-5, "c_draft": float(rng.uniform(0.01, 0.5)),
              "c_tree": 1e-7, "bucket_ratio": 0.0}
    n_max = 48
    obj = S.objectives(coeffs, lens, trees, n_max)
    peak = int(np.argmax(obj))
    assert all(obj[i] < obj[i - 1] for i in range(peak + 1, n_max)
               if obj[i] != obj[i - 1]), "objective not unimodal"
    n, seen = S.select(coeffs, lens, trees, n_max, patience=1)
    assert n == peak + 1


def test_cost_formula_and_buckets_by_hand():
    c = {"c0": 2.0, "c_seq": 0.001, "c_draft": 0.5, "c_tree": 0.0001, "bucket_ratio": 0.0}
    assert S.cost(c, 1000, 8, 8000) == pytest.approx(2.0 + 1.0 + 4.0 + 0.8)
    # octave buckets (r = 1): x = 5 lies in [4, 8), represented by 2^2.5
    c2 = dict(c, bucket_ratio=1.0)
    assert S.cost(c2, 5, 0, 0) == pytest.approx(2.0 + 0.001 * 2 ** 2.5)
    assert S.cost(c2, 4, 0, 0) == S.cost(c2, 7, 0, 0) != S.cost(c2, 8, 0, 0)
    assert S.cost(c2, 0, 0, 0) == 2.0


def test_fit_recovers_known_coefficients():
    rng = np.random.default_rng(3)
    truth = np.array([3.5, 2e-5, 0.02, 3e-8])
    rows = []
    for _ in range(30):
        ns, nd = float(rng.integers(1000, 700000)), float(rng.integers(1, 16384))
        tk = ns * float(rng.integers(1, 64))
        rows.append((ns, nd, tk, float(truth @ [1, ns, nd, tk])))
    assert np.allclose(S.fit(rows), truth, rtol=1e-6)


def test_planted_mistakes_are_caught():
    rng = np.random.default_rng(9)
    parents = random_tree(rng, 9)
    w = monotone_weights(rng, parents)

    def by_index(parents, w):          # ignores the weights
        return list(range(len(parents)))

    def lightest_first(parents, w):
        d = S.depths(parents)
        return [0] + sorted(range(1, len(parents)), key=lambda i: (w[i], d[i], i))

    for bad in (by_index, lightest_first):
        order = bad(parents, w)
        ok = all(math.isclose(sum(w[i] for i in order[:n]),
                              max(sum(w[i] for i in s) for s in connected_subsets(parents, n)))
                 for n in range(1, len(parents) + 1))
        assert not ok, bad.__name__
