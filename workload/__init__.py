"""Seeded synthetic inputs for the batched tree-verify step.

This module holds none of the verify arithmetic.  It only draws model
shapes, random weights, committed KV lengths, draft-tree topologies and
draft tokens, so that the HIP library and the oracle can be fed the very
same bits.  Where a draft is meant to follow the target model's greedy
choice, the caller supplies that choice through a callback.

The paper's own workloads (Llama-3.1-8B-Instruct with an EAGLE draft
model on LMSYS-Chat-1M and GSM8K prompts, Section 7.1) are not available;
these synthetic inputs stand in for them with the shapes, length
distributions and tree sizes of the verify step.
"""

from __future__ import annotations

import dataclasses
import heapq
import math
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_theta: float = 1e4
    rms_eps: float = 1e-5

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    def gemm_params(self) -> int:
        """Weights that enter a GEMM per token (embedding table excluded)."""
        H, d = self.hidden, self.head_dim
        per_layer = (H * (self.n_heads + 2 * self.n_kv_heads) * d + self.n_heads * d * H
                     + 3 * H * self.ffn)
        return self.n_layers * per_layer + self.vocab * H

    def kv_bytes_per_token(self) -> int:
        """bf16 K and V of one token over all layers."""
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim * 2


TINY = ModelConfig(n_layers=2, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=1024,
                   vocab=1024, rope_theta=1e4)
LLAMA_1B = ModelConfig(n_layers=16, hidden=2048, n_heads=32, n_kv_heads=8, head_dim=64, ffn=8192,
                       vocab=128256, rope_theta=5e5)
LLAMA_8B = ModelConfig(n_layers=32, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                       ffn=14336, vocab=128256, rope_theta=5e5)

WEIGHT_STD = 0.02


# ---------------------------------------------------------------------------
# Weights
# ---------------------------------------------------------------------------

def weight_shapes(cfg: ModelConfig):
    H, d, F = cfg.hidden, cfg.head_dim, cfg.ffn
    layer = [("attn_norm", (H,)), ("wq", (cfg.n_heads * d, H)), ("wk", (cfg.n_kv_heads * d, H)),
             ("wv", (cfg.n_kv_heads * d, H)), ("wo", (H, cfg.n_heads * d)), ("ffn_norm", (H,)),
             ("w_gate", (F, H)), ("w_up", (F, H)), ("w_down", (H, F))]
    return layer


def make_weights(cfg: ModelConfig, seed: int, device="cpu", dtype=torch.bfloat16):
    """Random weights: every matrix i.i.d. N(0, 0.02^2) drawn in float32 and
    then rounded to ``dtype`` (round to nearest even for bfloat16); every norm
    gain is 1.  Returns {"tok_embed", "final_norm", "lm_head", "layers": [...]}
    with the matrices in [out_features, in_features] layout.
    """
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))

    def randn(shape):
        t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
        t.mul_(WEIGHT_STD)
        return t.to(dtype)

    def ones(shape):
        return torch.ones(shape, device=device, dtype=dtype)

    W = {"tok_embed": randn((cfg.vocab, cfg.hidden)), "layers": []}
    for _ in range(cfg.n_layers):
        lw = {}
        for name, shape in weight_shapes(cfg):
            lw[name] = ones(shape) if name.endswith("norm") else randn(shape)
        W["layers"].append(lw)
    W["final_norm"] = ones((cfg.hidden,))
    W["lm_head"] = randn((cfg.vocab, cfg.hidden))
    return W


def prefix_kv_std(cfg: ModelConfig) -> float:
    """Scale of synthetic committed K/V: what an N(0, 0.02^2) projection of a
    unit-RMS hidden state produces, 0.02 * sqrt(hidden)."""
    return WEIGHT_STD * math.sqrt(cfg.hidden)


def fill_prefix_kv(view_k: torch.Tensor, view_v: torch.Tensor, S: int, std: float, gen):
    """Fill positions [0, S) of one sample's K and V views ([L, nkv, cap, d])
    with i.i.d. N(0, std^2) values rounded to the views' dtype."""
    if S == 0:
        return
    shape = view_k[:, :, :S].shape
    for view in (view_k, view_v):
        t = torch.randn(shape, generator=gen, device=view.device, dtype=torch.float32)
        t.mul_(std)
        view[:, :, :S].copy_(t.to(view.dtype))


# ---------------------------------------------------------------------------
# Lengths
# ---------------------------------------------------------------------------

def uniform_lengths(rng: np.random.Generator, B: int, lo: int, hi: int) -> np.ndarray:
    return rng.integers(lo, hi + 1, size=B).astype(np.int32)


def lognormal_lengths(rng: np.random.Generator, B: int, median: float, sigma: float,
                      lo: int, hi: int) -> np.ndarray:
    x = np.exp(rng.normal(math.log(median), sigma, size=B))
    return np.clip(np.rint(x), lo, hi).astype(np.int32)


# ---------------------------------------------------------------------------
# Tree topologies: parents[] in a topological order (parents[0] == -1)
# ---------------------------------------------------------------------------

def chain_tree(T: int) -> List[int]:
    return [-1] + list(range(T - 1))


def renumber_topological(parents: Sequence[int], rng: np.random.Generator) -> List[int]:
    """Relabel the nodes in a uniformly drawn topological order (root stays 0)."""
    T = len(parents)
    children = [[] for _ in range(T)]
    for i in range(1, T):
        children[parents[i]].append(i)
    order = [0]
    frontier = list(children[0])
    while frontier:
        j = int(rng.integers(len(frontier)))
        node = frontier.pop(j)
        order.append(node)
        frontier.extend(children[node])
    new_id = {old: new for new, old in enumerate(order)}
    out = [-1] * T
    for old in range(1, T):
        out[new_id[old]] = new_id[parents[old]]
    return out


def full_tree(levels: int, branching: int, rng: Optional[np.random.Generator] = None) -> List[int]:
    """Complete ``branching``-ary tree with ``levels`` levels (root = level 1)."""
    parents = [-1]
    level = [0]
    for _ in range(levels - 1):
        nxt = []
        for p in level:
            for _ in range(branching):
                parents.append(p)
                nxt.append(len(parents) - 1)
        level = nxt
    return renumber_topological(parents, rng) if rng is not None else parents


def level_tree(level_sizes: Sequence[int], rng: np.random.Generator) -> List[int]:
    """Tree with the given number of nodes per level; each node hangs from a
    uniformly drawn node of the previous level."""
    parents = [-1]
    prev = [0]
    for size in level_sizes[1:]:
        cur = []
        for _ in range(size):
            parents.append(prev[int(rng.integers(len(prev)))])
            cur.append(len(parents) - 1)
        prev = cur
    return renumber_topological(parents, rng)


def early_tree(rng: np.random.Generator, nodes: int = 8, levels: int = 4, width: int = 3) -> List[int]:
    """``nodes`` nodes on ``levels`` levels, at most ``width`` per level below the root."""
    rest = nodes - 1
    while True:
        sizes = rng.integers(1, width + 1, size=levels - 1)
        if int(sizes.sum()) == rest:
            break
    return level_tree([1] + [int(s) for s in sizes], rng)


def recursive_tree(rng: np.random.Generator, nodes: int, levels: int, max_children: int) -> List[int]:
    """Random recursive tree: a spine reaching ``levels`` levels, then every
    further node attaches to a uniformly drawn node that is not on the last
    level and has fewer than ``max_children`` children."""
    if not 1 <= levels <= nodes:
        raise ValueError("need 1 <= levels <= nodes")
    parents = [-1]
    depth = [0]
    nchild = [0]
    for lvl in range(1, levels):
        parents.append(lvl - 1)
        depth.append(lvl)
        nchild.append(0)
        nchild[lvl - 1] += 1
    while len(parents) < nodes:
        cand = [i for i in range(len(parents)) if depth[i] < levels - 1 and nchild[i] < max_children]
        if not cand:
            raise ValueError("tree is full at this depth and branching")
        p = cand[int(rng.integers(len(cand)))]
        parents.append(p)
        depth.append(depth[p] + 1)
        nchild.append(0)
        nchild[p] += 1
    return renumber_topological(parents, rng)


def draft_logit_tree(rng: np.random.Generator, n: int, levels: int = 8, branching: int = 4):
    """Top-``n`` connected selection by draft logit (Section 2.2).

    A candidate tree of ``levels`` levels and ``branching`` children per node
    gets sibling scores o(.) ~ Dirichlet(1) sorted in decreasing order; the
    draft logit of a node is the product of o over the non-root nodes of its
    branch (the root's own factor taken as 1).  The ``n`` nodes of largest
    draft logit are kept (ties: shallower, then earlier drawn).  Since the
    draft logit never grows along a branch, best-first expansion yields them
    and the set is connected.  Returns (parents, draft_logits).
    """
    parents, dls = [], []
    heap = [(-1.0, 0, 0, -1)]     # (-dl, depth, tiebreak, parent id)
    counter = 1
    while heap and len(parents) < n:
        negdl, dep, _, par = heapq.heappop(heap)
        node = len(parents)
        parents.append(par)
        dls.append(-negdl)
        if dep < levels - 1:
            o = np.sort(rng.dirichlet(np.ones(branching)))[::-1]
            for c in range(branching):
                heapq.heappush(heap, (negdl * float(o[c]), dep + 1, counter, node))
                counter += 1
    return parents, dls


def tree_depths(parents: Sequence[int]) -> List[int]:
    depth = [0] * len(parents)
    for i in range(1, len(parents)):
        depth[i] = depth[parents[i]] + 1
    return depth


def deepest_branch(parents: Sequence[int], rng: np.random.Generator) -> List[int]:
    """Node ids of the branch root -> a uniformly drawn deepest node."""
    depth = tree_depths(parents)
    dmax = max(depth)
    leaves = [i for i, dd in enumerate(depth) if dd == dmax]
    node = leaves[int(rng.integers(len(leaves)))]
    path = []
    while node != -1:
        path.append(node)
        node = parents[node] if node != 0 else -1
    return path[::-1]


# ---------------------------------------------------------------------------
# Tokens
# ---------------------------------------------------------------------------

def random_tokens(rng: np.random.Generator, T: int, vocab: int) -> List[int]:
    return [int(t) for t in rng.integers(0, vocab, size=T)]


def follow_greedy(trees, branches, p_follow: float, greedy_fn: Callable, rng: np.random.Generator):
    """Make each sample's designated branch follow the target's greedy choice.

    ``trees[b] = (tokens, parents)`` (tokens are modified in place);
    ``branches[b]`` is the branch root -> node to steer.  Level by level, the
    node at level l of the branch gets the greedy token after its parent with
    probability ``p_follow`` and keeps its random token otherwise.
    ``greedy_fn(trees)`` returns, per sample, the greedy token after every
    node; it is called once per level.
    """
    depth = max(len(br) for br in branches)
    coins = [rng.random(len(br)) for br in branches]
    for lvl in range(1, depth):
        if not any(len(br) > lvl for br in branches):
            break
        g = greedy_fn(trees)
        for b, br in enumerate(branches):
            if len(br) > lvl and coins[b][lvl] < p_follow:
                trees[b][0][br[lvl]] = int(g[b][br[lvl - 1]])
    return trees


# ---------------------------------------------------------------------------
# The five workloads
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    name: str
    cfg: ModelConfig
    seq_lens: np.ndarray               # committed length per sample
    trees: list                        # (tokens, parents) per sample
    branches: list                     # designated greedy-following branch per sample
    p_follow: float
    seed: int
    prompts: Optional[list] = None     # tiny workload: prompt tokens per sample

    @property
    def batch(self) -> int:
        return len(self.trees)

    @property
    def n_tokens(self) -> int:
        return sum(len(t[0]) for t in self.trees)


def _rngs(seed: int, n: int):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(n)]


def tiny_workload(seed: int = 0, batch: int = 4, prompt_len: int = 128, chain: int = 4) -> Workload:
    """2-layer decoder, 4 samples with a uniform 128-token prompt each, a
    chain draft of ``chain`` nodes (root + drafts); drafts follow greedy
    with p = 0.7 (each replaced by a random token with p = 0.3).  The root
    token is the greedy token after the prompt, filled in by the caller."""
    r_len, r_tree, r_tok = _rngs(seed, 3)
    prompts = [random_tokens(r_len, prompt_len, TINY.vocab) for _ in range(batch)]
    trees = [(random_tokens(r_tok, chain, TINY.vocab), chain_tree(chain)) for _ in range(batch)]
    branches = [list(range(chain)) for _ in range(batch)]
    return Workload("tiny", TINY, np.full(batch, prompt_len, np.int32), trees, branches, 0.7,
                    seed, prompts)


def llama1b_workload(seed: int = 1000, batch: int = 32) -> Workload:
    """1B shape; KV lengths U[512, 2048]; full binary 4-level tree (15 nodes)
    with random numbering; one deepest branch follows greedy with p = 0.7."""
    r_len, r_tree, r_tok = _rngs(seed, 3)
    lens = uniform_lengths(r_len, batch, 512, 2048)
    trees, branches = [], []
    for _ in range(batch):
        par = full_tree(4, 2, r_tree)
        trees.append((random_tokens(r_tok, len(par), LLAMA_1B.vocab), par))
        branches.append(deepest_branch(par, r_tree))
    return Workload("llama1b", LLAMA_1B, lens, trees, branches, 0.7, seed)


def early_workload(seed: int = 2000, batch: int = 128) -> Workload:
    """8B early-generation phase: KV lengths lognormal (median 1024, sigma
    0.8, clipped to [128, 8192]); 8-node trees on 4 levels, width <= 3."""
    r_len, r_tree, r_tok = _rngs(seed, 3)
    lens = lognormal_lengths(r_len, batch, 1024, 0.8, 128, 8192)
    trees, branches = [], []
    for _ in range(batch):
        par = early_tree(r_tree)
        trees.append((random_tokens(r_tok, len(par), LLAMA_8B.vocab), par))
        branches.append(deepest_branch(par, r_tree))
    return Workload("early", LLAMA_8B, lens, trees, branches, 0.7, seed)


def tail_workload(seed: int = 3000, batch: int = 4) -> Workload:
    """8B long-tail phase: 4 samples, KV lengths U[16384, 32768]; 64-node
    trees reaching 8 levels with at most 4 children per node."""
    r_len, r_tree, r_tok = _rngs(seed, 3)
    lens = uniform_lengths(r_len, batch, 16384, 32768)
    trees, branches = [], []
    for _ in range(batch):
        par = recursive_tree(r_tree, 64, 8, 4)
        trees.append((random_tokens(r_tok, len(par), LLAMA_8B.vocab), par))
        branches.append(deepest_branch(par, r_tree))
    return Workload("tail", LLAMA_8B, lens, trees, branches, 0.7, seed)


SWEEP_BATCHES = (1, 4, 16, 64, 256)
SWEEP_BUDGETS = (1, 4, 8, 16, 32, 64)


def sweep_lengths(seed: int = 4000, pool: int = 256) -> np.ndarray:
    """One pool of 256 KV lengths, lognormal (median 2048, sigma 0.8, clipped
    to [128, 16384]); a batch-B cell uses the first B samples."""
    (r_len,) = _rngs(seed, 1)
    return lognormal_lengths(r_len, pool, 2048, 0.8, 128, 16384)


def sweep_workload(batch: int, budget: int, seed: int = 4000) -> Workload:
    """Strategy-cost sweep cell: trees are the top-``budget`` draft-logit
    selections of a depth-8, branching-4 candidate tree."""
    lens = sweep_lengths(seed)[:batch]
    _, r_tree, r_tok = _rngs(seed + 7919 * budget, 3)
    trees, branches = [], []
    for _ in range(batch):
        par, _dl = draft_logit_tree(r_tree, budget)
        trees.append((random_tokens(r_tok, len(par), LLAMA_8B.vocab), par))
        branches.append(deepest_branch(par, r_tree))
    return Workload(f"sweep_b{batch}_n{budget}", LLAMA_8B, lens, trees, branches, 0.7, seed)
