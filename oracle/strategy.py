"""Oracle for the workload-aware drafting-strategy selection.

TEST INFRASTRUCTURE ONLY.  The plain statement of what the library's
cost predictor and draft-token-num selection compute; only the test suite
may import it.  It shares no code with the product path.

Paper, Section 5:
* objective (5.1): the draft token num n maximising al(n) / t_sd(n);
* al (5.2): the sum of the node weights w(u) = F(dl(u)) over the selected
  nodes (the root included, as in the paper's worked example where the
  root's weight is part of the sum);
* t_sd (5.2): a regression on N_seq (summed committed lengths) and N_draft
  (summed draft-token counts); the library adds the summed tree-size x
  committed-length product as a third feature (the attention work that
  grows with both).  Bucket cache: feature values in one bucket share one
  prediction;
* search (5.3): S(n+1) = S(n) plus the heaviest unselected node (principle
  2), within the first n layers (principle 1); the search over n stops once
  the objective keeps falling (early stopping justified by the sugar-water
  inequality).

Readings taken (the paper gives no formula for them):
* the selected set is the same n for every sample of the batch (the draft
  token num is one parameter of the step), capped by each tree's size;
* equal weights are ordered by depth, then node index;
* bucket b >= 1 of a feature x > 0 is floor(log(x) / log(1 + r)) + 1, bucket
  0 holds x = 0, and a bucket's prediction is the model at the geometric
  midpoint exp((b - 1/2) log(1 + r));
* early stopping: after `patience` consecutive strict falls of the
  objective; the answer is the first n of the largest objective seen.
"""

import math


def depths(parents):
    d = []
    for i, p in enumerate(parents):
        d.append(0 if p < 0 else d[p] + 1)
    return d


def selection_order(parents, w):
    """Nodes in the order they join S: the root, then the others by weight
    (heavier first), then depth, then index.  Because a child never weighs
    more than its parent, every prefix is a connected tree (principles 1, 2)."""
    d = depths(parents)
    rest = sorted(range(1, len(parents)), key=lambda i: (-w[i], d[i], i))
    return [0] + rest


def cost(coeffs, n_seq, n_draft, tree_kv):
    """t_sd in ms: c0 + c_seq N_seq + c_draft N_draft + c_tree TK, through the
    bucket rule when bucket_ratio > 0."""
    r = coeffs.get("bucket_ratio", 0.0)

    def rep(x):
        if r <= 0 or x <= 0:
            return float(x)
        lr = math.log1p(r)
        b = math.floor(math.log(x) / lr) + 1
        return math.exp((b - 0.5) * lr)

    return (coeffs["c0"] + coeffs["c_seq"] * rep(n_seq) + coeffs["c_draft"] * rep(n_draft) +
            coeffs["c_tree"] * rep(tree_kv))


def objectives(coeffs, seq_lens, trees, n_max):
    """al(n) / t_sd(n) for n = 1 .. n_max; trees = [(parents, w), ...]."""
    out = []
    orders = [selection_order(p, w) for p, w in trees]
    for n in range(1, n_max + 1):
        al = 0.0
        n_seq = n_draft = tk = 0
        for (p, w), order, S in zip(trees, orders, seq_lens):
            k = min(n, len(p))
            al += sum(w[i] for i in order[:k])
            n_seq += S
            n_draft += k
            tk += k * S
        out.append(al / cost(coeffs, n_seq, n_draft, tk))
    return out


def select(coeffs, seq_lens, trees, n_max, patience):
    """The draft token num the search returns, and the objectives it saw."""
    obj = objectives(coeffs, seq_lens, trees, n_max)
    best_n, best, falls, seen = 1, -1.0, 0, []
    for n in range(1, n_max + 1):
        o = obj[n - 1]
        seen.append(o)
        if o > best:
            best, best_n = o, n
        falls = falls + 1 if n > 1 and o < obj[n - 2] else 0
        if falls >= patience:
            break
    return best_n, seen


def fit(rows):
    """Coefficients (c0, c_seq, c_draft, c_tree) of t_sd minimising the summed
    squared relative error over measured steps: rows of (n_seq, n_draft,
    tree_kv, ms).  Plain weighted normal equations in float64 (weight
    1 / ms^2)."""
    import numpy as np
    X = np.array([[1.0, r[0], r[1], r[2]] for r in rows])
    y = np.array([r[3] for r in rows])
    W = np.diag(1.0 / y ** 2)
    return np.linalg.solve(X.T @ W @ X, X.T @ W @ y)
