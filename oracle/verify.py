"""Oracle for one batched speculative-decoding tree-verify step.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously
correct CPU statement of what the verify step computes.  Only the test
suite, the package smoke check and the benchmark's CPU-baseline leg may
import or call it; the product path (the HIP library and its Python
binding) never does, and shares no code, table or helper with it.

Everything is computed with plain PyTorch CPU operations in float64.
Weights and KV-cache entries may be handed in in any floating dtype
(bfloat16 in practice); they are upcast to float64 before use.

What is computed (paper, Section 2.2 "Speculative Decoding"; Section 5.2
names the two costs of verification, attention over the KV cache and the
FFN matrix products; Section 6.2 states that a verify step leaves the
previously verified KV cache untouched):

* Each sample carries a committed prefix of ``S_b`` tokens whose K/V are
  already cached, and a draft token tree whose node 0 (the root) is the
  token decided by the previous step.  Every node is a token, every
  root-to-node branch a candidate continuation.
* Node ``i`` sits at position ``S_b + depth(i)`` and sees the whole
  prefix plus its own ancestors (itself included) in the tree: exactly the
  causal view it would have if its branch were decoded on its own.
* The target model is a Llama-style decoder (RMSNorm, rotary position
  embedding, grouped-query attention, SwiGLU feed-forward, untied LM
  head).  The logits of node ``i`` are the next-token logits after its
  branch.
* Greedy acceptance (temperature 0): ``g_i = argmax`` of node ``i``'s
  logits (lowest id on ties).  A node is accepted when every edge on its
  branch carries the token the parent predicted; the root is always
  accepted.  The deepest accepted node (lowest index on ties) is ``best``;
  ``accepted_len = depth(best)`` and ``next_token = g_best``.
* The K/V entries of the nodes on the path root -> best then occupy cache
  positions ``S_b .. S_b + accepted_len`` and the committed length grows
  by ``accepted_len + 1``.

Readings of points the paper leaves open are listed with the function
that applies them.

Precision.  By default every step is exact float64 arithmetic: the plain
definition.  ``operand_dtype=torch.bfloat16`` instead rounds every operand
of every matrix product to bfloat16 (RMSNorm outputs, q/k/v, the softmax
numerators, the attention output, the SwiGLU activation; weights and cached
K/V already are bfloat16) and keeps everything else exact.  That is an ideal
bf16-operand computation of the same definition; the tests use it only to
measure how far bf16 storage alone moves the logits of a deep random-weight
model, which sets the tolerance for full-depth comparisons.  It is pinned
against an independent decoder with the same storage points rounded (the
Hugging Face Llama in float64 with rounding hooks, each branch decoded on its
own), and each of its rounding points is shown to matter by a planted
omission.
"""

from __future__ import annotations

import math

import torch

F64 = torch.float64


def _f64(t: torch.Tensor) -> torch.Tensor:
    return t.detach().to(device="cpu", dtype=F64)


# ---------------------------------------------------------------------------
# Tree bookkeeping (Section 2.2: node = token, branch = candidate sequence)
# ---------------------------------------------------------------------------

def tree_metadata(parents):
    """Depth of every node and its ancestor set (itself included).

    Reading: nodes arrive in a topological order, ``parents[0] == -1`` and
    ``0 <= parents[i] < i`` otherwise; the root has depth 0.
    Returns ``depth`` (int64 [T]) and ``anc`` (bool [T, T]) with
    ``anc[i, j]`` true iff node ``j`` lies on the branch root -> ``i``.
    """
    T = len(parents)
    if T < 1 or int(parents[0]) != -1:
        raise ValueError("node 0 must be the root (parent -1)")
    depth = [0] * T
    anc = torch.zeros(T, T, dtype=torch.bool)
    anc[0, 0] = True
    for i in range(1, T):
        p = int(parents[i])
        if not 0 <= p < i:
            raise ValueError(f"node {i} has parent {p}; need 0 <= parent < node")
        depth[i] = depth[p] + 1
        anc[i] = anc[p]
        anc[i, i] = True
    return torch.tensor(depth, dtype=torch.int64), anc


def greedy_accept(tokens, parents, g):
    """Greedy tree acceptance (Section 2.2, read at temperature 0).

    ``g[i]`` is the target's greedy token after node ``i``.  Returns
    ``(accepted_len, next_token, path)``: ``path`` lists the node indices of
    the branch root -> best in depth order, so ``len(path) ==
    accepted_len + 1``.
    """
    T = len(tokens)
    depth, _ = tree_metadata(parents)
    accepted = [False] * T
    accepted[0] = True
    for i in range(1, T):
        p = int(parents[i])
        accepted[i] = accepted[p] and int(tokens[i]) == int(g[p])
    best = 0
    for i in range(T):
        if accepted[i] and depth[i] > depth[best]:
            best = i
    path = []
    node = best
    while node != -1:
        path.append(node)
        node = int(parents[node]) if node != 0 else -1
    path.reverse()
    return int(depth[best]), int(g[best]), path


# ---------------------------------------------------------------------------
# Model pieces (Llama-style decoder)
# ---------------------------------------------------------------------------

def rms_norm(x: torch.Tensor, gain: torch.Tensor, eps: float) -> torch.Tensor:
    """x / sqrt(mean(x^2) + eps) * gain, over the last axis."""
    return x * torch.rsqrt((x * x).mean(dim=-1, keepdim=True) + eps) * gain


def rope_cos_sin(pos: torch.Tensor, head_dim: int, theta: float):
    """cos/sin of the rotation angles, float64.

    Reading (rotary embedding, not specified by the paper): frequency
    ``j`` (0 <= j < head_dim/2) is ``theta ** (-2 j / head_dim)`` and the
    angle of position ``p`` is ``p * freq_j``; no frequency rescaling.
    """
    half = head_dim // 2
    freq = torch.tensor([theta ** (-2.0 * j / head_dim) for j in range(half)], dtype=F64)
    ang = pos.to(F64)[:, None] * freq[None, :]
    return torch.cos(ang), torch.sin(ang)


def rope(x: torch.Tensor, cos: torch.Tensor, sin: torch.Tensor) -> torch.Tensor:
    """Rotate ``x`` [n, heads, d] in the half-split convention.

    Element ``j`` of the first half pairs with element ``j + d/2``:
    (a, b) -> (a cos - b sin, b cos + a sin).
    """
    half = x.shape[-1] // 2
    a, b = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return torch.cat([a * c - b * s, b * c + a * s], dim=-1)


def _identity(t):
    return t


def attention(q, k_all, v_all, visible, n_kv_heads, rnd=_identity):
    """Masked softmax attention for one sample.

    q: [T, nq, d]; k_all, v_all: [nkv, S+T, d]; visible: bool [T, S+T].
    Query head ``h`` reads KV head ``h // (nq / nkv)`` (grouped-query
    attention).  Scores are scaled by 1/sqrt(d); the softmax is
    exp(s - max s) / sum exp(s - max s), and ``rnd`` is applied to its
    numerators where they enter the product with V.
    """
    T, nq, d = q.shape
    group = nq // n_kv_heads
    out = torch.zeros(T, nq, d, dtype=F64)
    for h in range(nq):
        kv = h // group
        s = (q[:, h, :] @ k_all[kv].T) / math.sqrt(d)
        s = s.masked_fill(~visible, float("-inf"))
        e = torch.exp(s - s.max(dim=-1, keepdim=True).values)
        out[:, h, :] = (rnd(e) @ v_all[kv]) / e.sum(dim=-1, keepdim=True)
    return out


def forward(cfg, W, samples, operand_dtype=None):
    """Target-model forward over the nodes of several samples.

    ``samples`` is a list of dicts with keys ``tokens`` (list[int]),
    ``pos`` (int64 [T]), ``visible_tree`` (bool [T, T]: which of the
    sample's new tokens each one sees), ``prefix_k``/``prefix_v``
    ([L, nkv, S, d]; S may be 0).  Every new token sees the whole prefix.

    Returns the float64 logits [sum T, V] and, per sample, the new tokens'
    post-rotation keys and values [L, nkv, T, d].  ``operand_dtype``: see the
    module docstring.
    """
    if operand_dtype is None:
        rnd = _identity
    else:
        def rnd(t):
            return t.to(operand_dtype).to(F64)
    L, nq, nkv, d = cfg.n_layers, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    tokens = [t for s in samples for t in s["tokens"]]
    starts = []
    n = 0
    for s in samples:
        starts.append(n)
        n += len(s["tokens"])
    N = n
    pos = torch.cat([s["pos"] for s in samples]).to(torch.int64)
    cos, sin = rope_cos_sin(pos, d, cfg.rope_theta)

    x = _f64(W["tok_embed"])[torch.tensor(tokens, dtype=torch.int64)]
    new_k = [torch.zeros(L, nkv, len(s["tokens"]), d, dtype=F64) for s in samples]
    new_v = [torch.zeros(L, nkv, len(s["tokens"]), d, dtype=F64) for s in samples]

    for l in range(L):
        lw = W["layers"][l]
        h = rnd(rms_norm(x, _f64(lw["attn_norm"]), cfg.rms_eps))
        q = (h @ _f64(lw["wq"]).T).view(N, nq, d)
        k = (h @ _f64(lw["wk"]).T).view(N, nkv, d)
        v = rnd((h @ _f64(lw["wv"]).T).view(N, nkv, d))
        q = rnd(rope(q, cos, sin))
        k = rnd(rope(k, cos, sin))
        o = torch.zeros(N, nq, d, dtype=F64)
        for b, s in enumerate(samples):
            lo, T = starts[b], len(s["tokens"])
            kb = k[lo:lo + T].transpose(0, 1)          # [nkv, T, d]
            vb = v[lo:lo + T].transpose(0, 1)
            new_k[b][l] = kb
            new_v[b][l] = vb
            pk = _f64(s["prefix_k"][l]) if s["prefix_k"] is not None else torch.zeros(nkv, 0, d, dtype=F64)
            pv = _f64(s["prefix_v"][l]) if s["prefix_v"] is not None else torch.zeros(nkv, 0, d, dtype=F64)
            S = pk.shape[1]
            k_all = torch.cat([pk, kb], dim=1)
            v_all = torch.cat([pv, vb], dim=1)
            visible = torch.cat([torch.ones(T, S, dtype=torch.bool), s["visible_tree"]], dim=1)
            o[lo:lo + T] = attention(q[lo:lo + T], k_all, v_all, visible, nkv, rnd)
        x = x + rnd(o.reshape(N, nq * d)) @ _f64(lw["wo"]).T
        h2 = rnd(rms_norm(x, _f64(lw["ffn_norm"]), cfg.rms_eps))
        gate = h2 @ _f64(lw["w_gate"]).T
        up = h2 @ _f64(lw["w_up"]).T
        x = x + rnd(torch.nn.functional.silu(gate) * up) @ _f64(lw["w_down"]).T

    hf = rnd(rms_norm(x, _f64(W["final_norm"]), cfg.rms_eps))
    logits = hf @ _f64(W["lm_head"]).T
    return logits, new_k, new_v


# ---------------------------------------------------------------------------
# The verify step, its commit, and a prefill built from the same forward
# ---------------------------------------------------------------------------

def verify(cfg, W, prefix_k, prefix_v, seq_lens, trees, operand_dtype=None):
    """One batched tree-verify step.

    prefix_k[b], prefix_v[b]: committed K/V of sample b, [L, nkv, >= S_b, d]
    (positions S_b onward are ignored).  seq_lens[b] = S_b.
    trees[b] = (tokens, parents).

    Returns a dict with per-node ``logits`` (float64 [N, V]), ``argmax``
    (int64 [N]), ``depth``, ``pos``, per-sample ``anc`` (bool [T, T]),
    ``accepted_len``, ``next_token``, ``path`` and the new nodes' K/V
    (``tree_k``/``tree_v``, [L, nkv, T, d] per sample).
    """
    samples = []
    depths, ancs = [], []
    for b, (tokens, parents) in enumerate(trees):
        if len(tokens) != len(parents):
            raise ValueError("tokens and parents differ in length")
        for t in tokens:
            if not 0 <= int(t) < cfg.vocab:
                raise ValueError(f"token {t} out of range")
        depth, anc = tree_metadata(parents)
        S = int(seq_lens[b])
        depths.append(depth)
        ancs.append(anc)
        pk = prefix_k[b][:, :, :S] if prefix_k is not None and prefix_k[b] is not None else None
        pv = prefix_v[b][:, :, :S] if prefix_v is not None and prefix_v[b] is not None else None
        if S > 0 and (pk is None or pk.shape[2] != S):
            raise ValueError("prefix K/V shorter than seq_len")
        samples.append({"tokens": [int(t) for t in tokens], "pos": S + depth,
                        "visible_tree": anc, "prefix_k": pk, "prefix_v": pv})
    logits, new_k, new_v = forward(cfg, W, samples, operand_dtype)
    g = torch.argmax(logits, dim=-1)   # first maximal index = lowest id on ties

    acc_len, nxt, paths = [], [], []
    off = 0
    for b, (tokens, parents) in enumerate(trees):
        T = len(tokens)
        a, n, p = greedy_accept(tokens, parents, g[off:off + T].tolist())
        acc_len.append(a)
        nxt.append(n)
        paths.append(p)
        off += T
    return {
        "logits": logits,
        "argmax": g,
        "depth": torch.cat(depths),
        "pos": torch.cat([s["pos"] for s in samples]),
        "anc": ancs,
        "accepted_len": acc_len,
        "next_token": nxt,
        "path": paths,
        "tree_k": new_k,
        "tree_v": new_v,
    }


def commit(prefix_k, prefix_v, seq_lens, result, cache_dtype=torch.bfloat16):
    """Append each sample's accepted path to its committed K/V.

    The verified prefix is never rewritten (Section 6.2, the Markov property
    of verification).  The cache stores ``cache_dtype``, so the appended
    entries are rounded to it.  Returns new (prefix_k, prefix_v, seq_lens).
    """
    out_k, out_v, out_s = [], [], []
    for b, path in enumerate(result["path"]):
        S = int(seq_lens[b])
        idx = torch.tensor(path, dtype=torch.int64)
        add_k = result["tree_k"][b][:, :, idx].to(cache_dtype)
        add_v = result["tree_v"][b][:, :, idx].to(cache_dtype)
        pk = prefix_k[b][:, :, :S].to(cache_dtype)
        pv = prefix_v[b][:, :, :S].to(cache_dtype)
        out_k.append(torch.cat([pk, add_k], dim=2))
        out_v.append(torch.cat([pv, add_v], dim=2))
        out_s.append(S + len(path))
    return out_k, out_v, out_s


def prefill(cfg, W, prompt, cache_dtype=torch.bfloat16, operand_dtype=None):
    """K/V of a prompt: the prompt is a chain whose every token sees all
    earlier ones (causal), starting at position 0.  Returns (K, V, logits)
    with K, V of shape [L, nkv, len(prompt), d] rounded to ``cache_dtype``.
    ``operand_dtype``: as for ``forward``.
    """
    T = len(prompt)
    causal = torch.tril(torch.ones(T, T, dtype=torch.bool))
    s = {"tokens": [int(t) for t in prompt], "pos": torch.arange(T, dtype=torch.int64),
         "visible_tree": causal, "prefix_k": None, "prefix_v": None}
    logits, ks, vs = forward(cfg, W, [s], operand_dtype)
    return ks[0].to(cache_dtype), vs[0].to(cache_dtype), logits
