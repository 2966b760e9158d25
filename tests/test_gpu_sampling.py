"""GPU parity of the acceptance variants (spec_verify_sampled) against the
oracle (oracle.sampling), through the C ABI.

Inputs are built so that both outcomes of every decision occur: the tree's
tokens are filled in level by level, each node's children drawn i.i.d. from
a draft q_u that mixes the target's own p_u (read from the GPU's logits of
the previous level) with a random distribution.

Comparison rule: the oracle runs on the very fp32 logits the library
sampled from (the debug dump), with the same draft rows and uniforms.
Accepted path and next token must be identical wherever every decision's
margin (relative distance of the acceptance test from its threshold,
distance of the uniform from the chosen CDF interval's edges) exceeds
1e-11; below that the two fp64 computations may round to different sides,
and only validity is checked.  Greedy acceptance with EOS takes integer
inputs and is bit-exact.
"""

import numpy as np
import pytest
import torch

import paper_2512_04752_amd as sv
import workload as wl
from oracle import sampling as SA
from tests.gpu_util import (cpu_weights, device_setup, release, run_gpu, say, shallow,
                            split_rows, tiny_setup)

pytestmark = pytest.mark.gpu

MARGIN = 1e-11
U_MAX = np.float32(1.0 - 2.0 ** -24)


def depths_of(parents):
    d = []
    for p in parents:
        d.append(0 if p < 0 else d[p] + 1)
    return d


def fill_tokens_by_level(ver, ids, trees, lens, T, mix, seed, anti=False):
    """Draw every non-root token from its parent's q = mix p + (1 - mix) r
    (p the target at temperature T from the GPU's logits, r a random
    softmax, or with ``anti`` softmax(-3 z / T), a draft that favours the
    target's least likely tokens); returns the draft rows q [N, V] (fp32,
    on the device)."""
    V = ver.cfg.vocab
    offs = split_rows(trees)
    N = offs[-1]
    rng = np.random.default_rng(seed)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    q_all = torch.zeros(N, V, dtype=torch.float32, device="cuda")
    dep = [depths_of(t[1]) for t in trees]
    for d in range(max(max(x) for x in dep) + 1):
        out_dbg = ver.debug_buffers(N, logits=True)
        ver.verify(ids, trees, lens, debug=out_dbg)
        torch.cuda.synchronize()
        rows = [offs[b] + i for b, t in enumerate(trees) for i in range(len(t[0])) if dep[b][i] == d]
        ridx = torch.tensor(rows, device="cuda")
        z = out_dbg["logits"][ridx].double()
        p = torch.softmax(z / T, dim=1)
        if anti:
            r = torch.softmax(-3.0 * z / T, dim=1)
        else:
            r = torch.softmax(torch.randn(len(rows), V, generator=gen, device="cuda",
                                          dtype=torch.float64) * 2.0, dim=1)
        q = mix * p + (1.0 - mix) * r
        q = (q / q.sum(dim=1, keepdim=True)).float()
        q_all[ridx] = q
        cdf = torch.cumsum(q.double(), dim=1)
        row_of = {g: j for j, g in enumerate(rows)}
        kids = [(b, i) for b, t in enumerate(trees) for i in range(1, len(t[0]))
                if dep[b][i] == d + 1]
        if not kids:
            del out_dbg
            break
        src = torch.tensor([row_of[offs[b] + trees[b][1][i]] for b, i in kids], device="cuda")
        u = torch.tensor(rng.uniform(0, 1, len(kids)), device="cuda", dtype=torch.float64)
        tok = torch.searchsorted(cdf[src], (u * cdf[src, -1]).unsqueeze(1)).squeeze(1)
        tok = tok.clamp(max=V - 1).cpu().tolist()
        for (b, i), x in zip(kids, tok):
            trees[b][0][i] = int(x)
        del out_dbg
    return q_all


def uniforms_for(N, seed):
    u = np.random.default_rng(seed).uniform(0, 1, (N, 2)).astype(np.float32)
    return np.minimum(u, U_MAX)


def check_sampled(trees, out, q_all, U, T, eos, samples=None):
    """Oracle on the GPU's logits for ``samples`` (all by default); returns
    (exact, excused, accepted, rejected) counts."""
    offs = split_rows(trees)
    T32 = float(np.float32(T))
    exact = excused = accepted = rejected = 0
    for b in (range(len(trees)) if samples is None else samples):
        toks, pars = trees[b]
        sl = slice(offs[b], offs[b + 1])
        z = out["logits"][sl].double().numpy()
        q = q_all[sl].double().cpu().numpy()
        a, nx, path, margin = SA.sample_accept(toks, pars, z, T32, q, U[sl].astype(np.float64),
                                               eos=eos)
        g_len, g_next = out["accepted_len"][b], out["next_token"][b]
        g_nodes = out["nodes"][b].tolist()
        g_path = g_nodes[:g_len + 1]
        assert all(x == -1 for x in g_nodes[g_len + 1:])
        if margin > MARGIN:
            assert (g_len, g_next, g_path) == (a, nx, path), \
                f"sample {b}: gpu {(g_len, g_next, g_path)} oracle {(a, nx, path)} margin {margin}"
            exact += 1
        else:
            excused += 1
            assert g_path[0] == 0 and all(pars[g_path[k + 1]] == g_path[k] for k in range(g_len))
            assert -1 <= g_next < len(q[0])
        accepted += a > 0
        # a rejection happened where a node on the path has children and the
        # walk did not move to the first of them
        rejected += any(SA.children(pars, u) and (k + 1 == len(path) or
                                                  path[k + 1] != SA.children(pars, u)[0])
                        for k, u in enumerate(path))
    return exact, excused, accepted, rejected


def random_parents(rng, n, max_children=4):
    parents, kids = [-1], [0]
    for i in range(1, n):
        p = int(rng.choice([j for j in range(i) if kids[j] < max_children]))
        parents.append(p)
        kids[p] += 1
        kids.append(0)
    return parents


@pytest.mark.parametrize("T", [0.5, 1.0, 2.0])
def test_tiny_sampled_matches_oracle(T):
    say(f"tiny model, 16 samples, random trees of 1..40 nodes, T = {T}")
    cfg, w, W_cpu, W_dev, ver = tiny_setup(seed=4, batch=16, extra_cap=64, sampling=True)
    rng = np.random.default_rng(70)
    trees = []
    for b in range(w.batch):
        par = random_parents(rng, int(rng.integers(1, 41)))
        trees.append(([w.trees[b][0][0]] + [0] * (len(par) - 1), par))
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    q_all = fill_tokens_by_level(ver, ids, trees, lens, T, mix=0.6, seed=71)
    N = sum(len(t[0]) for t in trees)
    U = uniforms_for(N, 72)
    dbg = ver.debug_buffers(N, logits=True)
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, T, -1, q_all,
                                         torch.from_numpy(U).cuda(), debug=dbg)
    torch.cuda.synchronize()
    out = {"logits": dbg["logits"].cpu(), "accepted_len": acc.cpu().tolist(),
           "next_token": nxt.cpu().tolist(), "nodes": nodes.cpu()}
    exact, excused, accepted, rejected = check_sampled(trees, out, q_all, U, T, -1)
    say(f"  exact {exact}, excused {excused}, samples with accepts {accepted}, "
        f"with a rejection {rejected}")
    assert exact >= 15 and accepted > 0 and rejected > 0
    release(ver, W_dev)


def test_tiny_sampled_large_trees():
    """T = 1 over trees past one 64-bit ancestor word: random trees of 256,
    130 and 65 nodes and a root with 199 children (far more rejected
    children than the recomputed residuals cover, so the walk continues on
    the stored residual row)."""
    cfg, w, W_cpu, W_dev, ver = tiny_setup(seed=8, batch=4, extra_cap=256, sampling=True,
                                           max_tokens=4 * 256)
    rng = np.random.default_rng(98)
    pars = [random_parents(rng, 256), random_parents(rng, 130), [-1] + [0] * 199,
            random_parents(rng, 65)]
    trees = [([w.trees[b][0][0]] + [0] * (len(p) - 1), p) for b, p in enumerate(pars)]
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    q_all = fill_tokens_by_level(ver, ids, trees, lens, 1.0, mix=0.6, seed=99)
    N = sum(len(t[0]) for t in trees)
    U = uniforms_for(N, 100)
    dbg = ver.debug_buffers(N, logits=True)
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, 1.0, -1, q_all,
                                         torch.from_numpy(U).cuda(), debug=dbg)
    torch.cuda.synchronize()
    out = {"logits": dbg["logits"].cpu(), "accepted_len": acc.cpu().tolist(),
           "next_token": nxt.cpu().tolist(), "nodes": nodes.cpu()}
    exact, excused, accepted, rejected = check_sampled(trees, out, q_all, U, 1.0, -1)
    say(f"  exact {exact}, excused {excused}, accepted lengths {out['accepted_len']}")
    assert exact + excused == len(trees) and exact >= 3
    release(ver, W_dev)


def rejections(pars, path):
    """Children rejected at each node of an accepted path (the oracle's walk):
    those before the taken child, all of them at the last node."""
    out = []
    for k, u in enumerate(path):
        kids = SA.children(pars, u)
        out.append(kids.index(path[k + 1]) if k + 1 < len(path) else len(kids))
    return out


def test_tiny_sampled_wide_star():
    """Roots with 20 to 40 children drawn from a draft that favours the
    target's least likely tokens: nodes with more than eight rejected
    children continue on the stored residual row."""
    cfg, w, W_cpu, W_dev, ver = tiny_setup(seed=7, batch=8, extra_cap=64, sampling=True)
    rng = np.random.default_rng(95)
    trees = []
    for b in range(w.batch):
        n = int(rng.integers(21, 42))
        par = [-1] + [0] * (n - 1)
        if b % 2:                                   # a second level under the first child
            par = par[:n - 6] + [1] * 6
        trees.append(([w.trees[b][0][0]] + [0] * (n - 1), par))
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    q_all = fill_tokens_by_level(ver, ids, trees, lens, 1.0, mix=0.02, seed=96, anti=True)
    N = sum(len(t[0]) for t in trees)
    U = uniforms_for(N, 97)
    dbg = ver.debug_buffers(N, logits=True)
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, 1.0, -1, q_all,
                                         torch.from_numpy(U).cuda(), debug=dbg)
    torch.cuda.synchronize()
    out = {"logits": dbg["logits"].cpu(), "accepted_len": acc.cpu().tolist(),
           "next_token": nxt.cpu().tolist(), "nodes": nodes.cpu()}
    exact, excused, accepted, rejected = check_sampled(trees, out, q_all, U, 1.0, -1)
    most = 0
    for b, (toks, pars) in enumerate(trees):
        L = out["accepted_len"][b]
        most = max(most, max(rejections(pars, out["nodes"][b][:L + 1].tolist())))
    say(f"  exact {exact}, excused {excused}, most rejections at one node {most}")
    assert exact >= 7 and most > 8
    release(ver, W_dev)


def test_tiny_sampled_with_eos():
    """T = 1 with an EOS token taken from an accepted node of sample 0, and
    sample 1's root set to EOS."""
    cfg, w, W_cpu, W_dev, ver = tiny_setup(seed=5, batch=8, extra_cap=64, sampling=True)
    rng = np.random.default_rng(80)
    trees = []
    for b in range(w.batch):
        par = random_parents(rng, int(rng.integers(4, 30)), max_children=2)
        trees.append(([w.trees[b][0][0]] + [0] * (len(par) - 1), par))
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    q_all = fill_tokens_by_level(ver, ids, trees, lens, 1.0, mix=0.9, seed=81)
    N = sum(len(t[0]) for t in trees)
    U = uniforms_for(N, 82)
    # first pass without EOS: pick the EOS token from an accepted non-root node
    dbg = ver.debug_buffers(N, logits=True)
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, 1.0, -1, q_all,
                                         torch.from_numpy(U).cuda(), debug=dbg)
    torch.cuda.synchronize()
    lens_acc = acc.cpu().tolist()
    cands = [b for b in range(w.batch) if b != 1 and lens_acc[b] >= 1 and
             trees[b][0][int(nodes[b, 1])] != trees[b][0][0]]
    assert cands, "no sample accepted a node"
    b0 = cands[0]
    eos = trees[b0][0][int(nodes[b0, 1])]
    trees[1][0][0] = eos
    say(f"  EOS token {eos} (accepted at depth 1 of sample {b0})")
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, 1.0, eos, q_all,
                                         torch.from_numpy(U).cuda(), debug=dbg)
    torch.cuda.synchronize()
    out = {"logits": dbg["logits"].cpu(), "accepted_len": acc.cpu().tolist(),
           "next_token": nxt.cpu().tolist(), "nodes": nodes.cpu()}
    check_sampled(trees, out, q_all, U, 1.0, eos)
    assert out["accepted_len"][1] == 0 and out["next_token"][1] == -1
    assert out["next_token"][b0] == -1 and out["accepted_len"][b0] == 1
    release(ver, W_dev)


def greedy_chains(ver, ids, trees, lens, p_follow, rng):
    """Set each chain node's token to its parent's greedy successor with
    probability p_follow (level by level from the GPU's argmax)."""
    offs = split_rows(trees)
    depth = max(len(t[0]) for t in trees)
    for d in range(1, depth):
        out = run_gpu(ver, ids, trees, lens, logits=False)
        g = out["argmax"].tolist()
        for b, (toks, pars) in enumerate(trees):
            if d < len(toks) and rng.random() < p_follow:
                toks[d] = g[offs[b] + pars[d]]


def test_tiny_greedy_with_eos_large_trees():
    """Greedy acceptance with EOS on chains of up to 256 nodes that follow the
    GPU's greedy choice: one accepted to its end (past depth 64), one cut
    where its greedy token equals the EOS token, one by a wrong token at node
    90; the oracle's rule on the GPU's own argmax, bitwise."""
    cfg, w, W_cpu, W_dev, ver = tiny_setup(seed=9, batch=3, extra_cap=256, sampling=True,
                                           max_tokens=3 * 256)
    rng = np.random.default_rng(91)
    sizes = [120, 200, 256]
    trees = [([w.trees[b][0][0]] + [0] * (n - 1), list(range(-1, n - 1))) for b, n in enumerate(sizes)]
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    greedy_chains(ver, ids, trees, lens, 1.0, rng)
    # EOS: chain 1's greedy token at the first node from 100 on that chain 0 never
    # carries (greedy chains of a small model can cycle), so chain 0 runs to its end;
    # failing that, a token no chain carries
    seen0 = set(trees[0][0])
    pick = [i for i in range(100, 200) if trees[1][0][i] not in seen0]
    if pick:
        eos = int(trees[1][0][pick[0]])
    else:
        eos = min(set(range(cfg.vocab)) - set().union(*(set(t[0]) for t in trees)))
    trees[2][0][90] = (trees[2][0][90] + 1) % cfg.vocab
    offs = split_rows(trees)
    dbg = ver.debug_buffers(offs[-1], logits=False)
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, 0.0, eos, None, None, debug=dbg)
    torch.cuda.synchronize()
    g = dbg["argmax"].cpu().tolist()
    lens_got = []
    for b, (toks, pars) in enumerate(trees):
        want = SA.greedy_accept_eos(toks, pars, g[offs[b]:offs[b + 1]], eos)
        got_len = int(acc[b])
        got = (got_len, int(nxt[b]), nodes[b, :got_len + 1].cpu().tolist())
        assert got == want, f"sample {b}: gpu {got[:2]} oracle {want[:2]}"
        assert (nodes[b, got_len + 1:] == -1).all()
        lens_got.append(got_len)
    say(f"  accepted lengths {lens_got}")
    assert max(lens_got) > 64
    release(ver, W_dev)


def test_tiny_greedy_with_eos_is_bit_exact():
    """T = 0 with an EOS token: the oracle's greedy-with-EOS rule on the
    GPU's own argmax tokens; and with no EOS token, the sampled entry point
    at T = 0 equals plain spec_verify."""
    cfg, w, W_cpu, W_dev, ver = tiny_setup(seed=6, batch=8, extra_cap=64, sampling=True)
    rng = np.random.default_rng(90)
    trees = []
    for b in range(w.batch):
        n = int(rng.integers(3, 9))
        trees.append(([w.trees[b][0][0]] + [int(x) for x in rng.integers(0, cfg.vocab, n - 1)],
                      list(range(-1, n - 1))))
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    greedy_chains(ver, ids, trees, lens, 0.85, rng)
    offs = split_rows(trees)
    eos = trees[0][0][2]
    trees[3][0][0] = eos
    N = offs[-1]
    for e in (eos, -1):
        dbg = ver.debug_buffers(N, logits=False)
        acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, 0.0, e, None, None, debug=dbg)
        torch.cuda.synchronize()
        g = dbg["argmax"].cpu().tolist()
        for b, (toks, pars) in enumerate(trees):
            want = SA.greedy_accept_eos(toks, pars, g[offs[b]:offs[b + 1]], e)
            got_len = int(acc[b])
            got = (got_len, int(nxt[b]), nodes[b, :got_len + 1].cpu().tolist())
            assert got == want, f"sample {b}, eos {e}: gpu {got} oracle {want}"
            assert (nodes[b, got_len + 1:] == -1).all()
        if e == -1:
            plain = run_gpu(ver, ids, trees, lens, logits=False)
            assert plain["accepted_len"] == acc.cpu().tolist()
            assert plain["next_token"] == nxt.cpu().tolist()
            assert torch.equal(plain["nodes"], nodes.cpu())
    release(ver, W_dev)


@pytest.mark.parametrize("name,T", [("early", 1.0), ("tail", 0.7)])
def test_full_shape_sampled(name, T):
    """The Llama-8B shapes (vocab 128256, the early batch of 128 8-node trees
    and the tail batch of 4 64-node trees) on a two-layer model: the
    acceptance kernel sees the real vocabulary and tree sizes; the oracle
    checks a sample of the batch one by one."""
    make = {"early": wl.early_workload, "tail": wl.tail_workload}[name]
    w = shallow(make())
    say(f"{name}: sampled acceptance at T = {T}, batch {w.batch}, {w.n_tokens} nodes")
    W_dev = wl.make_weights(w.cfg, 60, device="cuda")
    ver = device_setup(w, W_dev, seed=6, sampling=True)
    ids, lens = list(range(w.batch)), w.seq_lens.tolist()
    trees = [(list(t[0]), list(t[1])) for t in w.trees]
    q_all = fill_tokens_by_level(ver, ids, trees, lens, T, mix=0.7, seed=61)
    say("  tokens drawn level by level")
    N = w.n_tokens
    U = uniforms_for(N, 62)
    dbg = ver.debug_buffers(N, logits=True)
    acc, nxt, nodes = ver.verify_sampled(ids, trees, lens, T, -1, q_all,
                                         torch.from_numpy(U).cuda(), debug=dbg)
    torch.cuda.synchronize()
    check = sorted(set([0, w.batch - 1] + [int(x) for x in
                                            np.random.default_rng(63).integers(0, w.batch, 6)]))
    offs = split_rows(trees)
    rows = torch.cat([torch.arange(offs[b], offs[b + 1]) for b in check])
    sub = [trees[b] for b in check]
    out = {"logits": dbg["logits"][rows.cuda()].cpu(),
           "accepted_len": [int(acc[b]) for b in check],
           "next_token": [int(nxt[b]) for b in check], "nodes": nodes[check].cpu()}
    exact, excused, accepted, rejected = check_sampled(sub, out, q_all[rows.cuda()],
                                                       U[rows.numpy()], T, -1)
    say(f"  checked {check}: exact {exact}, excused {excused}, accepts {accepted}, "
        f"rejections {rejected}")
    assert exact >= len(check) - 1
    # every sample: a valid path and a token in range
    for b, (toks, pars) in enumerate(trees):
        L = int(acc[b])
        path = nodes[b, :L + 1].tolist()
        assert path[0] == 0 and all(pars[path[k + 1]] == path[k] for k in range(L))
        assert 0 <= int(nxt[b]) < w.cfg.vocab
    release(ver, W_dev)
