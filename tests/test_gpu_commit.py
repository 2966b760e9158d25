"""GPU parity of KV compaction (spec_kv_commit) against the oracle's commit,
through the C ABI, on accepted branches deeper and wider than the verify tests
reach: whole chains of the largest tree, branches that jump over most of the tree, and
batches large enough that one work-group moves every K/V head of a layer in
several passes.  Pools hold random bit patterns, so a misplaced element cannot
match by accident; the comparison is bitwise."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2512_04752_amd as sv
import workload as wl
from tests.gpu_util import say
from tests.test_gpu_transfer import random_pool, views

pytestmark = pytest.mark.gpu

MAX_TREE = sv.SPEC_MAX_TREE


def random_branch(rng, depth):
    """Node ids of an accepted branch with ``depth`` accepted drafts: 0, then
    distinct increasing ids, so node path[d] >= d as in a topologically
    numbered tree (the branch is a chain of parent links in some tree)."""
    if depth == 0:
        return [0]
    kind = rng.integers(3)
    if kind == 0:                       # straight chain: nothing moves
        return list(range(depth + 1))
    if kind == 1:                       # deepest ids: every row moves
        return [0] + list(range(MAX_TREE - depth, MAX_TREE))
    ids = np.sort(rng.choice(np.arange(1, MAX_TREE), size=depth, replace=False))
    return [0] + [int(x) for x in ids]


CASES = {
    # (config, batch, seed).  At the 8B shape batch 40 puts all 16 K/V heads of
    # a layer in one work-group (a branch as deep as the largest tree takes many passes) and batch 4
    # two heads; the 2-layer and tiny cases give one head per work-group.
    "llama8b_b40": (wl.LLAMA_8B, 40, 0),
    "llama8b_b4": (wl.LLAMA_8B, 4, 1),
    "llama1b_2layer_b5": (dataclasses.replace(wl.LLAMA_1B, n_layers=2), 5, 2),
    "tiny_b4": (wl.TINY, 4, 3),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_commit_matches_oracle_bitwise(name):
    cfg, batch, seed = CASES[name]
    rng = np.random.default_rng(seed)
    n_pool = batch + 1                  # one sample stays out of the commit
    lens = rng.integers(1, 48, size=n_pool).tolist()
    caps = [S + MAX_TREE + int(rng.integers(0, 8)) for S in lens]
    ids = rng.permutation(n_pool)[:batch].tolist()
    depths = [int(x) for x in rng.integers(0, MAX_TREE, size=batch)]
    depths[0], depths[-1] = MAX_TREE - 1, 0
    paths = [random_branch(rng, dd) for dd in depths]
    say(f"commit {name}: batch {batch}, depths {depths[:8]}...")

    pool = random_pool(cfg, caps, 100 + seed)
    ks, vs = views(pool, range(n_pool))
    seq = [lens[i] for i in ids]
    acc = torch.tensor(depths, dtype=torch.int32, device="cuda")
    nodes = torch.zeros(batch, MAX_TREE, dtype=torch.int32)
    for b, p in enumerate(paths):
        nodes[b, :len(p)] = torch.tensor(p, dtype=torch.int32)
    nodes = nodes.cuda()
    new_lens = torch.full((batch,), -1, dtype=torch.int32, device="cuda")
    sv.spec_kv_commit(pool, ids, seq, acc, nodes, new_lens)
    torch.cuda.synchronize()
    ks2, vs2 = views(pool, range(n_pool))

    # the oracle appends the K/V of the path's nodes (tree slots S + node) to
    # the committed prefix
    result = {"path": paths,
              "tree_k": [ks[i][:, :, lens[i]:lens[i] + MAX_TREE] for i in ids],
              "tree_v": [vs[i][:, :, lens[i]:lens[i] + MAX_TREE] for i in ids]}
    ek, ev, es = oracle.commit([ks[i] for i in ids], [vs[i] for i in ids], seq, result,
                               cache_dtype=torch.int16)
    assert new_lens.cpu().tolist() == es
    moved = 0
    for b, i in enumerate(ids):
        n = es[b]
        assert torch.equal(ks2[i][:, :, :n], ek[b]), f"K of sample {i}"
        assert torch.equal(vs2[i][:, :, :n], ev[b]), f"V of sample {i}"
        moved += sum(int(node != d) for d, node in enumerate(paths[b]))
    out = [i for i in range(n_pool) if i not in ids]
    for i in out:                       # not in the batch: untouched
        assert torch.equal(ks2[i], ks[i]) and torch.equal(vs2[i], vs[i])
    say(f"  rows moved {moved}")
    assert moved > 0
