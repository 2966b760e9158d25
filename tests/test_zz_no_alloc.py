"""spec_verify_noalloc, the verify step on the library's static device
scratch, against spec_verify on the same inputs through the C ABI: two calls
in a row, the second smaller than the first, each compared bitwise on every
output (accepted lengths, next tokens, accepted branches, logits, greedy
tokens, tree metadata) and on the tree K/V it writes into the pool."""

import dataclasses

import numpy as np
import pytest
import torch

import paper_2512_04752_amd as sv
import workload as wl
from tests.gpu_util import device_setup, release, say, tiny_setup

pytestmark = pytest.mark.gpu


def tree_slots(ver, ids, trees, lens):
    out = []
    for i, (t, S) in zip(ids, zip(trees, lens)):
        k, v = ver.kv.sample_view(int(i))
        out.append((k[:, :, S:S + len(t[0])].clone(), v[:, :, S:S + len(t[0])].clone()))
    return out


def scribble(ver, ids, trees, lens):
    for i, (t, S) in zip(ids, zip(trees, lens)):
        k, v = ver.kv.sample_view(int(i))
        k[:, :, S:S + len(t[0])].fill_(7.0)
        v[:, :, S:S + len(t[0])].fill_(-7.0)


def run(ver, ids, trees, lens, dbg, noalloc):
    fn = ver.verify_noalloc if noalloc else ver.verify
    acc, nxt, nodes = fn(ids, trees, lens, debug=dbg)
    torch.cuda.synchronize()
    res = {k: v.cpu() for k, v in dbg.items()}
    res.update(acc=acc.cpu(), nxt=nxt.cpu(), nodes=nodes.cpu())
    return res


def compare(ver, ids, trees, lens):
    n = sum(len(t[0]) for t in trees)
    a = run(ver, ids, trees, lens, ver.debug_buffers(n, logits=True), noalloc=False)
    ka = tree_slots(ver, ids, trees, lens)
    scribble(ver, ids, trees, lens)
    dbg = ver.debug_buffers(n, logits=True)
    for t in dbg.values():
        t.fill_(-1)
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    b = run(ver, ids, trees, lens, dbg, noalloc=True)
    free1 = torch.cuda.mem_get_info()[0]
    kb = tree_slots(ver, ids, trees, lens)
    for key in a:
        assert torch.equal(a[key], b[key]), key
    for (k1, v1), (k2, v2) in zip(ka, kb):
        assert torch.equal(k1, k2) and torch.equal(v1, v2)
    say(f"  {len(ids)} samples, {sum(len(t[0]) for t in trees)} nodes: bitwise equal; "
        f"device memory free before/after the call {free0 >> 20} / {free1 >> 20} MiB")
    return free0, free1


def test_noalloc_tiny_two_calls():
    say("noalloc: tiny model, 4 samples then 2")
    cfg, w, W_cpu, W_dev, ver = tiny_setup(3, extra_cap=64)
    rng = np.random.default_rng(3)
    ids, lens = list(range(4)), [int(x) for x in w.seq_lens]
    trees = [(wl.random_tokens(rng, n, cfg.vocab), wl.recursive_tree(rng, n, min(n, 6), 3))
             for n in (24, 5, 40, 1)]
    compare(ver, ids, trees, lens)
    # second call: smaller batch, other samples, other trees (stale scratch must not matter)
    trees2 = [(wl.random_tokens(rng, n, cfg.vocab), wl.recursive_tree(rng, n, min(n, 4), 3))
              for n in (9, 3)]
    _, free1 = compare(ver, [3, 1], trees2, [lens[3], lens[1]])
    _, free2 = compare(ver, [3, 1], trees2, [lens[3], lens[1]])
    assert free2 == free1     # a repeated call allocates nothing
    release(ver, W_dev)


def test_noalloc_8b_shape_two_calls():
    """2-layer 8B shape: the early workload (128 samples, 1024 nodes; split-KV
    partials and split-K partials in the scratch), then the tail workload's
    trees (4 samples x 64 nodes: the 8-wave attention kernel) on the first 4
    samples of the same pool."""
    w = wl.early_workload(2000)
    w.cfg = dataclasses.replace(w.cfg, n_layers=2)
    say(f"noalloc: 2-layer 8B shape, batch {w.batch}, {w.n_tokens} nodes, then 4 x 64 nodes")
    W_dev = wl.make_weights(w.cfg, 80, device="cuda")
    ver = device_setup(w, W_dev, cap_extra=64, seed=8)
    ids, lens = list(range(w.batch)), [int(x) for x in w.seq_lens]
    compare(ver, ids, w.trees, lens)
    t = wl.tail_workload(3000)
    compare(ver, [0, 1, 2, 3], t.trees, lens[:4])
    release(ver, W_dev)
