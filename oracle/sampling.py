"""Oracle for the acceptance variants of the verify step: speculative sampling
over the draft tree at a temperature T > 0, and greedy acceptance with an
end-of-sequence token.

TEST INFRASTRUCTURE ONLY.  A plain float64 statement of what the library's
sampled and EOS acceptance compute; only the test suite may import it.  It
shares no code with the product path.

Paper, Section 2.2: speculative decoding keeps the target model's output
distribution (the cited rejection-sampling proofs).  The paper never writes
the rule out for trees at T > 0; this statement takes the multi-draft form
of speculative sampling for a token tree, under these readings:

* the draft drew the children of node u independently from its distribution
  q_u (a row of ``draft_probs``, indexed by u); a child with token x is
  accepted with probability min(1, r(x) / q_u(x)), r being the current
  residual target distribution (at first r = p_u = softmax(z_u / T));
* children are tried in node order; a rejected child replaces r by
  max(r - q_u, 0) renormalised; the walk moves to the first accepted child;
* when no child is accepted (or u has none) the next token is drawn from r by
  inverse CDF: the smallest y whose cumulative mass exceeds the uniform;
* random numbers are inputs: ``uniforms[c][0]`` decides child c,
  ``uniforms[u][1]`` draws the next token after u;
* a residual whose mass is zero after a rejection (possible only through
  rounding, since a residual equal to q_u accepts every child) falls back
  to p_u;
* EOS: an accepted node carrying the end-of-sequence token ends its branch;
  its children are not considered and there is no next token (-1).
  A root carrying EOS accepts nothing.

Greedy acceptance with EOS is the greedy rule (a node is accepted when its
parent is and its token is the parent's argmax successor; the deepest
accepted node, lowest index on ties, ends the path) with accepted EOS nodes
accepting no children and giving no next token.
"""

import numpy as np


def softmax_t(z, temperature):
    """p = softmax(z / T) in float64."""
    x = np.asarray(z, dtype=np.float64) / float(temperature)
    x = x - x.max()
    e = np.exp(x)
    return e / e.sum()


def inverse_cdf(r, a):
    """The smallest index y with sum(r[:y+1]) > a (r normalised, a in [0, 1));
    the last index of positive mass when rounding leaves a at or above the
    total.  Also returns the decision's margin: the distance from a to the
    nearer edge of the chosen index's CDF interval."""
    c = np.cumsum(r)
    hit = np.nonzero(c > a)[0]
    if len(hit):
        y = int(hit[0])
    else:
        y = int(np.nonzero(r > 0)[0][-1])
    lo = c[y - 1] if y > 0 else 0.0
    return y, min(abs(a - lo), abs(c[y] - a))


def children(parents, u):
    return [c for c in range(len(parents)) if c > 0 and int(parents[c]) == u]


def sample_accept(tokens, parents, logits, temperature, draft_probs, uniforms, eos=-1):
    """Speculative-sampling acceptance over one sample's tree.

    tokens, parents: the tree (node 0 is the root, parents[0] = -1);
    logits: [T, V] target logits after every node; draft_probs: [T, V], row u
    the distribution u's children were drawn from; uniforms: [T, 2].
    Returns (accepted_len, next_token, path, margin): ``path`` the accepted
    node indices root first, ``margin`` the smallest distance of any decision
    from its threshold (relative for acceptance tests), for tie excusal.
    """
    z = np.asarray(logits, dtype=np.float64)
    q = np.asarray(draft_probs, dtype=np.float64)
    a = np.asarray(uniforms, dtype=np.float64)
    path, margin = [0], np.inf
    if int(tokens[0]) == eos:
        return 0, -1, path, margin
    u = 0
    while True:
        p = softmax_t(z[u], temperature)
        r = p.copy()
        moved = None
        for c in children(parents, u):
            x = int(tokens[c])
            # accept iff a < r(x) / q(x), written without the division so that
            # q(x) = 0 accepts exactly when r(x) > 0
            lhs, rhs = a[c, 0] * q[u, x], r[x]
            margin = min(margin, abs(rhs - lhs) / max(rhs, lhs, 1e-300))
            if lhs < rhs:
                moved = c
                break
            res = np.maximum(r - q[u], 0.0)
            tot = res.sum()
            r = res / tot if tot > 0 else p
        if moved is None:
            y, m = inverse_cdf(r, a[u, 1])
            return len(path) - 1, y, path, min(margin, m)
        u = moved
        path.append(u)
        if int(tokens[u]) == eos:
            return len(path) - 1, -1, path, margin


def greedy_accept_eos(tokens, parents, g, eos):
    """Greedy tree acceptance with an end-of-sequence token; g[i] is the
    argmax successor of node i.  Returns (accepted_len, next_token, path)."""
    n = len(tokens)
    depth = [0] * n
    accepted = [False] * n
    accepted[0] = True
    for i in range(1, n):
        p = int(parents[i])
        depth[i] = depth[p] + 1
        accepted[i] = accepted[p] and int(tokens[p]) != eos and int(tokens[i]) == int(g[p])
    if int(tokens[0]) == eos:
        accepted = [i == 0 for i in range(n)]
    best = 0
    for i in range(n):
        if accepted[i] and depth[i] > depth[best]:
            best = i
    path = [best]
    while path[-1] != 0:
        path.append(int(parents[path[-1]]))
    path.reverse()
    nxt = -1 if int(tokens[best]) == eos else int(g[best])
    return depth[best], nxt, path
