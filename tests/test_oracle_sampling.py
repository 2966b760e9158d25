"""Pins of the acceptance-variant oracle (oracle.sampling), CPU only.

* losslessness (Section 2.2): over many seeded trials of a tiny target and
  draft (children drawn i.i.d. from the draft), the first two emitted tokens
  follow the target's joint distribution (chi-square test);
* special cases: a draft equal to the target accepts every first child; at
  a vanishing temperature with distinct sibling tokens the walk is the
  greedy rule; a residual that runs dry falls back to the target;
* hand-computed steps: rejection, residual, inverse CDF;
* EOS: hand examples, and brute force over every branch of random trees;
  with no EOS token the EOS variant is the plain greedy rule;
* plausible mistakes planted in copies of the walk fail the chi-square test.
"""

import math

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import sampling as SA


def log(p):
    return np.log(np.asarray(p, dtype=np.float64))


# ---------------------------------------------------------------------------
# hand-computed steps
# ---------------------------------------------------------------------------

def test_reject_then_residual_by_hand():
    # p = (.5, .3, .2), q = (.2, .5, .3); child token 1: p/q = 0.6
    z = np.stack([log([0.5, 0.3, 0.2]), log([0.1, 0.1, 0.8])])
    q = np.array([[0.2, 0.5, 0.3], [1 / 3] * 3])
    toks, par = [2, 1], [-1, 0]
    # a = 0.7 > 0.6: rejected; residual max(p - q, 0) = (.3, 0, 0) -> token 0
    for a2 in (0.0, 0.5, 0.999):
        assert SA.sample_accept(toks, par, z, 1.0, q, [[0, a2], [0.7, 0.5]])[:3] == (0, 0, [0])
    # a = 0.5 < 0.6: accepted; node 1 has no children, next from p_1 = (.1, .1, .8)
    assert SA.sample_accept(toks, par, z, 1.0, q, [[0, 0], [0.5, 0.15]])[:3] == (1, 1, [0, 1])
    assert SA.sample_accept(toks, par, z, 1.0, q, [[0, 0], [0.5, 0.05]])[:3] == (1, 0, [0, 1])
    assert SA.sample_accept(toks, par, z, 1.0, q, [[0, 0], [0.5, 0.25]])[:3] == (1, 2, [0, 1])


def test_two_rejections_by_hand():
    # p = (.4, .3, .2, .1), q = (.1, .5, .1, .3); children tokens 3 then 3
    # first: p(3)/q(3) = 1/3, a = 0.5 rejects; r = (.3, 0, .1, 0)/.4 = (.75, 0, .25, 0)
    # second: r(3) = 0 rejects for any a; r = max(r - q, 0) = (.65, 0, .15, 0)/.8
    #   = (.8125, 0, .1875, 0); inverse CDF at 0.85 -> 2, at 0.5 -> 0
    z = np.stack([log([0.4, 0.3, 0.2, 0.1])] + [log([0.25] * 4)] * 2)
    q = np.array([[0.1, 0.5, 0.1, 0.3]] + [[0.25] * 4] * 2)
    toks, par = [0, 3, 3], [-1, 0, 0]
    U = np.array([[0, 0.85], [0.5, 0], [0.0, 0]])
    assert SA.sample_accept(toks, par, z, 1.0, q, U)[:3] == (0, 2, [0])
    U[0, 1] = 0.5
    assert SA.sample_accept(toks, par, z, 1.0, q, U)[:3] == (0, 0, [0])
    # a second child with token 2 instead: r(2)/q(2) = 2.5 accepts for any a
    assert SA.sample_accept([0, 3, 2], par, z, 1.0, q, [[0, 0], [0.5, 0], [0.99, 0.9]])[:3] \
        == (1, 3, [0, 2])


def test_temperature_scales_logits():
    # z = log p at T = 1; at T = 2 the target is p^(1/2) normalised
    p = np.array([0.64, 0.36])
    z = np.stack([log(p), log(p)])
    q = np.array([[0.5, 0.5], [0.5, 0.5]])
    # T = 2: p' = (.8, .6)/1.4 = (4/7, 3/7); child token 1: ratio 6/7
    res = SA.sample_accept([0, 1], [-1, 0], z, 2.0, q, [[0, 0], [0.85, 0.5]])
    assert res[:3] == (1, 0, [0, 1])
    res = SA.sample_accept([0, 1], [-1, 0], z, 2.0, q, [[0, 0], [0.86, 0.5]])
    assert res[:3] == (0, 0, [0])             # residual (1/7, 0) -> token 0
    assert SA.softmax_t(z[0], 2.0) == pytest.approx([4 / 7, 3 / 7], rel=1e-12)


def test_inverse_cdf_edges():
    assert SA.inverse_cdf(np.array([0.0, 0.5, 0.0, 0.5]), 0.0)[0] == 1
    assert SA.inverse_cdf(np.array([0.0, 0.5, 0.0, 0.5]), 0.5)[0] == 3
    assert SA.inverse_cdf(np.array([0.2, 0.3, 0.5, 0.0]), 0.999999)[0] == 2
    # a total rounded below a: the last index of positive mass
    assert SA.inverse_cdf(np.array([0.3, 0.3, 0.3999999, 0.0]), 0.99999999)[0] == 2


# ---------------------------------------------------------------------------
# special cases
# ---------------------------------------------------------------------------

def random_tree(rng, n, max_children=4):
    parents, kids = [-1], [0]
    for i in range(1, n):
        cands = [j for j in range(i) if kids[j] < max_children]
        p = int(rng.choice(cands))
        parents.append(p)
        kids[p] += 1
        kids.append(0)
    return parents


@pytest.mark.parametrize("seed", range(6))
def test_draft_equal_to_target_accepts_first_children(seed):
    rng = np.random.default_rng(seed)
    V, n = 11, int(rng.integers(2, 20))
    par = random_tree(rng, n)
    z = rng.normal(0, 2, (n, V))
    T = float(rng.uniform(0.3, 2.0))
    q = np.stack([SA.softmax_t(z[i], T) for i in range(n)])
    toks = [int(rng.integers(V)) for _ in range(n)]
    U = rng.uniform(0, 1, (n, 2))
    U[:, 0] = np.minimum(U[:, 0], 0.999)
    a, nx, path, _ = SA.sample_accept(toks, par, z, T, q, U)
    want, u = [0], 0
    while SA.children(par, u):
        u = SA.children(par, u)[0]
        want.append(u)
    assert path == want and a == len(want) - 1


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("eos", [-1, 3])
def test_vanishing_temperature_is_greedy(seed, eos):
    """Logit gaps >= 0.01 at T = 1e-4 make every target one-hot to within
    e^-100; with distinct sibling tokens the walk follows the argmax child,
    as the greedy rule does."""
    rng = np.random.default_rng(50 + seed)
    V, n = 40, int(rng.integers(1, 30))
    par = random_tree(rng, n)
    z = np.stack([rng.permutation(V) * 0.01 for _ in range(n)])
    g = z.argmax(axis=1)
    toks = [int(rng.integers(V))]
    for i in range(1, n):
        sib = {toks[c] for c in range(1, i) if par[c] == par[i]}
        # follow the argmax half of the time, else a fresh token
        x = int(g[par[i]]) if rng.random() < 0.5 else int(rng.integers(V))
        while x in sib:
            x = int(rng.integers(V))
        toks.append(x)
    q = rng.dirichlet(np.ones(V) * 0.5, n)
    U = rng.uniform(0, 1, (n, 2))
    a, nx, path, _ = SA.sample_accept(toks, par, z, 1e-4, q, U, eos=eos)
    assert (a, nx, path) == SA.greedy_accept_eos(toks, par, g, eos)
    if eos < 0:
        assert (a, nx, path) == oracle.greedy_accept(toks, par, g.tolist())


def test_dry_residual_falls_back_to_target():
    # q(1) = 1 and p = (.5, .5): child token 1 rejected (a = 0.6 > 0.5); the
    # residual max(p - q, 0) = (.5, 0) is not dry.  A q that covers p exactly
    # except on the rejected token cannot occur, so force the dry case with
    # q >= p everywhere (q not normalised): residual 0 -> draw from p.
    z = np.stack([log([0.5, 0.5]), log([0.5, 0.5])])
    q = np.array([[0.6, 0.6], [0.5, 0.5]])
    assert SA.sample_accept([0, 1], [-1, 0], z, 1.0, q, [[0, 0.7], [0.9, 0]])[:3] == (0, 1, [0])
    assert SA.sample_accept([0, 1], [-1, 0], z, 1.0, q, [[0, 0.3], [0.9, 0]])[:3] == (0, 0, [0])


# ---------------------------------------------------------------------------
# EOS
# ---------------------------------------------------------------------------

def test_eos_by_hand():
    toks, par, g = [5, 7, 9, 7], [-1, 0, 1, 0], [7, 9, 3, 2]
    assert SA.greedy_accept_eos(toks, par, g, eos=7) == (1, -1, [0, 1])
    assert SA.greedy_accept_eos(toks, par, g, eos=-1) == (2, 3, [0, 1, 2])
    assert SA.greedy_accept_eos(toks, par, g, eos=9) == (2, -1, [0, 1, 2])
    assert SA.greedy_accept_eos(toks, par, g, eos=5) == (0, -1, [0])
    # sampled: a draft equal to the target walks 0 -> 1 -> 2; EOS at node 1 stops there
    V = 10
    z = np.random.default_rng(0).normal(size=(3, V))
    q = np.stack([SA.softmax_t(r, 1.0) for r in z])
    U = np.full((3, 2), 0.5)
    assert SA.sample_accept([5, 7, 9], [-1, 0, 1], z, 1.0, q, U, eos=7)[:3] == (1, -1, [0, 1])
    assert SA.sample_accept([5, 7, 9], [-1, 0, 1], z, 1.0, q, U, eos=5)[:3] == (0, -1, [0])
    a, nx, path, _ = SA.sample_accept([5, 7, 9], [-1, 0, 1], z, 1.0, q, U, eos=4)
    assert (a, path) == (2, [0, 1, 2]) and nx >= 0


@pytest.mark.parametrize("seed", range(20))
def test_greedy_eos_by_brute_force(seed):
    """Every branch root..i is accepted iff each edge follows the parent's
    argmax and no node before i is EOS; the answer is the deepest accepted
    branch (lowest index on ties)."""
    rng = np.random.default_rng(900 + seed)
    V, n = 4, int(rng.integers(1, 25))
    par = random_tree(rng, n, max_children=3)
    toks = [int(x) for x in rng.integers(V, size=n)]
    g = [int(x) for x in rng.integers(V, size=n)]
    eos = int(rng.integers(-1, V))
    best, best_path = None, None
    for i in range(n):
        br = [i]
        while br[-1] != 0:
            br.append(par[br[-1]])
        br.reverse()
        ok = all(toks[br[k + 1]] == g[br[k]] for k in range(len(br) - 1)) and \
            all(toks[v] != eos for v in br[:-1])
        if ok and (best is None or len(br) > len(best_path)):
            best, best_path = i, br
    want_next = -1 if toks[best] == eos else g[best]
    assert SA.greedy_accept_eos(toks, par, g, eos) == (len(best_path) - 1, want_next, best_path)


# ---------------------------------------------------------------------------
# losslessness: the emitted tokens follow the target distribution
# ---------------------------------------------------------------------------

V_L = 5
TRIALS = 12000


def markov_pair(seed):
    """A target and a draft whose next-token distributions depend on the
    depth and the current token: logits Z[depth][token] and Q[depth][token]
    (the draft deliberately far from the target)."""
    rng = np.random.default_rng(seed)
    Z = rng.normal(0, 1.2, (3, V_L, V_L))
    Q = rng.dirichlet(np.ones(V_L) * 0.7, (3, V_L))
    return Z, Q


def emitted_pairs(walk, Z, Q, T, seed, shape=(3, 2)):
    """First two emitted tokens over TRIALS steps from root token 0: the
    accepted path's tokens then the next token; when a step emits one token
    the second comes from the target directly (the following step)."""
    rng = np.random.default_rng(seed)
    k0, k1 = shape
    par = [-1] + [0] * k0 + [1 + c for c in range(k0) for _ in range(k1)]
    depth = [0] + [1] * k0 + [2] * (k0 * k1)
    n = len(par)
    counts = np.zeros((V_L, V_L), dtype=np.int64)
    for _ in range(TRIALS):
        toks = [0] * n
        for i in range(1, n):
            p = par[i]
            toks[i] = int(rng.choice(V_L, p=Q[depth[p], toks[p]]))
        z = np.stack([Z[depth[i], toks[i]] for i in range(n)])
        q = np.stack([Q[depth[i], toks[i]] for i in range(n)])
        U = rng.uniform(0, 1, (n, 2))
        a, nx, path = walk(toks, par, z, T, q, U)[:3]
        out = [toks[i] for i in path[1:]] + [nx]
        if len(out) < 2:
            p1 = SA.softmax_t(Z[1, out[0]], T)
            out.append(int(rng.choice(V_L, p=p1)))
        counts[out[0], out[1]] += 1
    return counts


def exact_pairs(Z, T):
    p0 = SA.softmax_t(Z[0, 0], T)
    return np.array([[p0[x] * SA.softmax_t(Z[1, x], T)[y] for y in range(V_L)]
                     for x in range(V_L)])


def chi2_pvalue(counts, probs):
    exp = probs.ravel() * counts.sum()
    stat = ((counts.ravel() - exp) ** 2 / exp).sum()
    return stats.chi2.sf(stat, exp.size - 1)


@pytest.mark.slow
@pytest.mark.parametrize("T", [1.0, 0.6])
def test_emitted_tokens_follow_the_target(T):
    Z, Q = markov_pair(7)
    counts = emitted_pairs(SA.sample_accept, Z, Q, T, seed=11)
    assert chi2_pvalue(counts, exact_pairs(Z, T)) > 1e-4


def walk_with(mistake):
    """A copy of the walk with one plausible mistake."""

    def walk(toks, par, z, T, q, U):
        u, path = 0, [0]
        while True:
            p = SA.softmax_t(z[u], T)
            r = p.copy()
            moved = None
            for c in SA.children(par, u):
                x = toks[c]
                qq = q[c] if mistake == "child_q" else q[u]
                if mistake == "ignore_q":
                    ok = U[c, 0] < r[x]
                else:
                    ok = U[c, 0] * qq[x] < r[x]
                if ok:
                    moved = c
                    break
                if mistake == "no_residual":
                    continue
                res = np.maximum(r - qq, 0.0)
                r = res if mistake == "unnormalised" else res / res.sum()
            if moved is None:
                if mistake == "draw_from_target":
                    r = p
                y, _ = SA.inverse_cdf(r / r.sum(), U[u, 1])
                return len(path) - 1, y, path
            u = moved
            path.append(u)

    return walk


@pytest.mark.slow
@pytest.mark.parametrize("mistake", ["ignore_q", "no_residual", "unnormalised", "child_q",
                                     "draw_from_target"])
def test_planted_mistakes_fail_losslessness(mistake):
    Z, Q = markov_pair(7)
    counts = emitted_pairs(walk_with(mistake), Z, Q, 1.0, seed=11)
    assert chi2_pvalue(counts, exact_pairs(Z, 1.0)) < 1e-6, mistake


def test_correct_copy_matches_oracle():
    """The mistake harness without a mistake is the oracle (so a failing
    mistake test is the mistake's doing)."""
    rng = np.random.default_rng(3)
    Z, Q = markov_pair(7)
    for _ in range(200):
        n = int(rng.integers(1, 12))
        par = random_tree(rng, n, 3)
        toks = [int(x) for x in rng.integers(V_L, size=n)]
        z = rng.normal(size=(n, V_L))
        q = rng.dirichlet(np.ones(V_L), n)
        U = rng.uniform(0, 1, (n, 2))
        assert walk_with(None)(toks, par, z, 0.8, q, U) == SA.sample_accept(toks, par, z, 0.8, q,
                                                                            U)[:3]
