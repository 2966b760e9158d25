"""Shared pieces of the GPU parity tests: building a workload on the device,
running the oracle on the same bits, and the comparison rules.

Comparison rules (tolerance of the verify step on bf16 logits):
* shallow models (2 layers) at hidden <= 2048: |z_gpu - z_oracle| <= ATOL +
  RTOL * |z_oracle| element-wise against the exact oracle;
* deeper or wider models: bf16 storage noise alone moves random-weight
  logits further than that (the oracle's ideal bf16-operand computation,
  pinned on the CPU against an independently rounded decoder, misses it
  too), so the GPU's error against the exact oracle must stay inside the
  envelope of that ideal computation's error: mean, 99.9th percentile,
  per-node relative L2 and maximum error at most ENV_FACTOR times the
  ideal's (plus a small floor);
* greedy tokens: equal, or "tie-excused" where the exact oracle's logit of
  the GPU's choice is within the tie tolerance of the oracle's maximum.  The
  tie tolerance is ATOL for the element-wise rule; under the envelope it is
  twice the largest error the envelope allows, ENV_FACTOR times the ideal
  computation's maximum error (plus the floor): never the GPU's own error.
  The excused count is bounded by that of the ideal computation
  (EXCUSE_FACTOR times its disagreements with the exact oracle, plus
  EXCUSE_SLACK);
* acceptance: bit-exact against the oracle's acceptance run on the GPU's own
  greedy tokens for every sample, and end to end equal to the oracle's for
  every checked sample with no excused disagreement at a node that either
  side accepts (only those nodes' greedy tokens decide acceptance);
* depth, positions, ancestor sets, compacted KV positions: bit-exact.

Every comparison appends one summary line to PARITY_LOG; the test session
prints them at its end.
"""

import dataclasses
import gc
import sys
import time

import numpy as np
import torch

import oracle
import paper_2512_04752_amd as sv
import workload as wl

ATOL, RTOL = 3e-2, 2e-2
ENV_FACTOR = 1.5
ENV_FLOOR = {"mean": 1e-3, "q999": 5e-3, "rowrel": 1e-3, "max": 5e-3}
EXCUSE_FACTOR, EXCUSE_SLACK = 3, 4

PARITY_LOG = []


def log_parity(line):
    import os
    test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0].split("::")[-1]
    PARITY_LOG.append(f"{test}: {line}")
    say("  parity " + line)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def cpu_weights(W):
    return {"tok_embed": W["tok_embed"].cpu(), "final_norm": W["final_norm"].cpu(),
            "lm_head": W["lm_head"].cpu(),
            "layers": [{k: v.cpu() for k, v in lw.items()} for lw in W["layers"]]}


def prefix_for_oracle(ver, ids, lens):
    ks, vs = [], []
    for i, S in zip(ids, lens):
        k, v = ver.kv.sample_view(int(i))
        ks.append(k[:, :, :int(S)].cpu())
        vs.append(v[:, :, :int(S)].cpu())
    return ks, vs


def run_gpu(ver, ids, trees, lens, logits=True, rows=None):
    """One verify through the C ABI with debug dumps; returns host results
    (only the logits of ``rows``, when given)."""
    n = sum(len(t[0]) for t in trees)
    dbg = ver.debug_buffers(n, logits=logits)
    acc, nxt, nodes = ver.verify(ids, trees, lens, debug=dbg)
    torch.cuda.synchronize()
    out = {k: (v[rows] if k == "logits" and rows is not None else v).cpu() for k, v in dbg.items()}
    del dbg
    out["accepted_len"] = acc.cpu().tolist()
    out["next_token"] = nxt.cpu().tolist()
    out["nodes"] = nodes.cpu()
    return out


def split_rows(trees):
    offs = [0]
    for t in trees:
        offs.append(offs[-1] + len(t[0]))
    return offs


def check_logits(z_gpu, z_or, what=""):
    z_or = z_or.to(torch.float64)
    z_gpu = z_gpu.to(torch.float64)
    err = (z_gpu - z_or).abs()
    bound = ATOL + RTOL * z_or.abs()
    bad = (err > bound)
    rel = (err / z_or.abs().clamp_min(1e-3)).max().item()
    say(f"  logits {what}: max_abs {err.max().item():.3e} max_rel {rel:.3e} "
        f"violations {int(bad.sum())}/{bad.numel()}")
    assert not bad.any(), f"{what}: {int(bad.sum())} logits outside tolerance, max err {err.max()}"
    return {"rule": "element-wise", "max_abs": err.max().item(), "max_rel": rel,
            "strict": 0.0, "tie_tol": ATOL, "ideal_flips": None}


def check_envelope(z_gpu, z_or, z_ideal, what=""):
    """Full-depth rule: the GPU's deviation from the exact oracle is no larger
    than the ideal bf16-operand computation's, within ENV_FACTOR (plus
    ENV_FLOOR), in mean, 99.9th percentile, per-node relative L2 and maximum.
    Returns the comparison's statistics and its tie tolerance, which comes
    from the ideal computation only."""
    z_or = z_or.to(torch.float64)
    e_gpu = (z_gpu.to(torch.float64) - z_or).abs()
    e_ref = (z_ideal.to(torch.float64) - z_or).abs()
    rr = lambda e: (e.norm(dim=-1) / z_or.norm(dim=-1)).max().item()     # noqa: E731
    q = lambda e: torch.quantile(e.flatten()[:: max(1, e.numel() // 4_000_000)].float(),  # noqa: E731
                                 0.999).item()
    stats = {"mean": (e_gpu.mean().item(), e_ref.mean().item()),
             "q999": (q(e_gpu), q(e_ref)), "rowrel": (rr(e_gpu), rr(e_ref)),
             "max": (e_gpu.max().item(), e_ref.max().item())}
    bound = ATOL + RTOL * z_or.abs()
    strict = (e_gpu > bound).float().mean().item()
    strict_ideal = (e_ref > bound).float().mean().item()
    say(f"  logits {what} (gpu, ideal bf16): " +
        " ".join(f"{k} {a:.3e}/{b:.3e}" for k, (a, b) in stats.items()) +
        f"; strict-rule violations {strict:.4%} / {strict_ideal:.4%}")
    for k, f in ENV_FLOOR.items():
        a, b = stats[k]
        assert a <= ENV_FACTOR * b + f, f"{what}: {k} error {a:.4e} exceeds envelope {b:.4e}"
    g_or = torch.argmax(z_or, dim=-1)
    ideal_flips = int((torch.argmax(z_ideal.to(torch.float64), dim=-1) != g_or).sum())
    tie_tol = 2 * (ENV_FACTOR * stats["max"][1] + ENV_FLOOR["max"])
    return {"rule": "envelope", "max_abs": stats["max"][0], "ideal_max_abs": stats["max"][1],
            "mean": stats["mean"], "strict": strict, "strict_ideal": strict_ideal,
            "tie_tol": tie_tol, "ideal_flips": ideal_flips}


def check_argmax(g_gpu, z_or, tol=ATOL):
    """Returns the rows of tie-excused disagreements; fails on any other."""
    g_or = torch.argmax(z_or, dim=-1)
    excused = []
    for i in range(len(g_gpu)):
        if int(g_gpu[i]) != int(g_or[i]):
            row = z_or[i]
            assert row[int(g_gpu[i])] >= row.max() - tol, \
                f"node {i}: gpu {int(g_gpu[i])} vs oracle {int(g_or[i])}, margin " \
                f"{(row.max() - row[int(g_gpu[i])]).item():.4f} beyond the tie tolerance {tol:.4f}"
            excused.append(i)
    return excused


def accepted_set(tokens, parents, g):
    """Nodes accepted under greedy tokens g (the root always)."""
    acc = [True] + [False] * (len(tokens) - 1)
    for i in range(1, len(tokens)):
        acc[i] = acc[parents[i]] and int(tokens[i]) == int(g[parents[i]])
    return {i for i in range(len(tokens)) if acc[i]}


def check_sample_acceptance(tokens, parents, g_gpu_b, gpu_len, gpu_next, gpu_nodes,
                            or_res=None, b=None, g_or_b=None, excused_nodes=()):
    """Bit-exact: the oracle's acceptance on the GPU's greedy tokens equals the
    GPU's; and, when no excused node is accepted by either side, equal to the
    oracle's own result.  Returns True when the end-to-end comparison ran."""
    a, nx, path = oracle.greedy_accept(tokens, parents, g_gpu_b)
    assert (gpu_len, gpu_next) == (a, nx)
    nodes = gpu_nodes.tolist()
    assert nodes[:a + 1] == path and all(x == -1 for x in nodes[a + 1:])
    if or_res is None:
        return False
    deciding = accepted_set(tokens, parents, g_gpu_b) | accepted_set(tokens, parents, g_or_b)
    if deciding & set(excused_nodes):
        return False
    assert or_res["accepted_len"][b] == a and or_res["path"][b] == path
    assert or_res["next_token"][b] == nx
    return True


def check_meta(trees, lens, out):
    offs = split_rows(trees)
    for b, (tokens, parents) in enumerate(trees):
        depth, anc = oracle.tree_metadata(parents)
        sl = slice(offs[b], offs[b + 1])
        assert out["depth"][sl].tolist() == depth.tolist()
        assert out["pos"][sl].tolist() == (int(lens[b]) + depth).tolist()
        bits = [sum(1 << j for j in range(len(parents)) if anc[i, j]) for i in range(len(parents))]
        # word w of a node holds nodes 64w .. 64w + 63
        got = [sum((int(x) & ((1 << 64) - 1)) << (64 * w) for w, x in enumerate(words))
               for words in out["anc"][sl].tolist()]
        assert got == bits


def full_check(cfg, W_cpu, ver, ids, trees, lens, check_ids=None, envelope=False):
    """GPU verify of the whole batch; oracle on samples ``check_ids`` (all by
    default).  ``envelope`` selects the full-depth rule.  Returns (gpu
    result, oracle result, excused count)."""
    offs = split_rows(trees)
    if check_ids is None:
        check_ids = list(range(len(trees)))
    rows = torch.cat([torch.arange(offs[b], offs[b + 1]) for b in check_ids])
    t0 = time.time()
    out = run_gpu(ver, ids, trees, lens, rows=rows)
    say(f"  gpu verify done ({time.time() - t0:.1f}s)")
    check_meta(trees, lens, out)
    g_gpu = out["argmax"].tolist()
    # acceptance on the GPU's own greedy tokens: every sample, bit-exact
    for b, (tokens, parents) in enumerate(trees):
        check_sample_acceptance(tokens, parents, g_gpu[offs[b]:offs[b + 1]],
                                out["accepted_len"][b], out["next_token"][b], out["nodes"][b])
    pk, pv = prefix_for_oracle(ver, [ids[b] for b in check_ids], [lens[b] for b in check_ids])
    t0 = time.time()
    r = oracle.verify(cfg, W_cpu, pk, pv, [lens[b] for b in check_ids],
                      [trees[b] for b in check_ids])
    say(f"  oracle on {len(check_ids)} samples done ({time.time() - t0:.1f}s)")
    if envelope:
        t0 = time.time()
        ri = oracle.verify(cfg, W_cpu, pk, pv, [lens[b] for b in check_ids],
                           [trees[b] for b in check_ids], operand_dtype=torch.bfloat16)
        say(f"  ideal bf16-operand oracle done ({time.time() - t0:.1f}s)")
        st = check_envelope(out["logits"], r["logits"], ri["logits"], f"{len(rows)} rows")
        del ri
    else:
        st = check_logits(out["logits"], r["logits"], f"{len(rows)} rows")
    excused = check_argmax(out["argmax"][rows], r["logits"], st["tie_tol"])
    if st["ideal_flips"] is not None:
        assert len(excused) <= EXCUSE_FACTOR * st["ideal_flips"] + EXCUSE_SLACK, \
            f"{len(excused)} excused disagreements, the ideal bf16 computation has {st['ideal_flips']}"
    roffs = split_rows([trees[b] for b in check_ids])
    g_or = r["argmax"].tolist()
    e2e = 0
    for j, b in enumerate(check_ids):
        tokens, parents = trees[b]
        exc_local = [i - roffs[j] for i in excused if roffs[j] <= i < roffs[j + 1]]
        e2e += check_sample_acceptance(tokens, parents, g_gpu[offs[b]:offs[b + 1]],
                                       out["accepted_len"][b], out["next_token"][b],
                                       out["nodes"][b], r, j, g_or[roffs[j]:roffs[j + 1]],
                                       exc_local)
    line = (f"L{cfg.n_layers} H{cfg.hidden} rows {len(rows)} {st['rule']}: "
            f"max_abs {st['max_abs']:.3g}")
    if st["rule"] == "envelope":
        line += (f" (ideal {st['ideal_max_abs']:.3g}), mean {st['mean'][0]:.3g} "
                 f"(ideal {st['mean'][1]:.3g}), strict-rule outside {st['strict']:.3%} "
                 f"(ideal {st['strict_ideal']:.3%})")
    line += (f", tie_tol {st['tie_tol']:.3g}, excused {len(excused)}"
             + (f" (ideal flips {st['ideal_flips']})" if st["ideal_flips"] is not None else "")
             + f", end-to-end {e2e}/{len(check_ids)} samples")
    log_parity(line)
    return out, r, len(excused)


def check_tree_kv(cfg, ver, ids, trees, lens, r, check_ids, layers=None):
    """K/V the verify wrote at slots S_b + node equal the oracle's (strict
    tolerance; ``layers`` limits the check, e.g. to the first layer of a
    deep model, whose K/V carry no accumulated bf16 noise)."""
    for j, b in enumerate(check_ids):
        k, v = ver.kv.sample_view(int(ids[b]))
        S, T = int(lens[b]), len(trees[b][0])
        sl = slice(None) if layers is None else slice(0, layers)
        kg = k[sl, :, S:S + T].cpu().to(torch.float64)
        vg = v[sl, :, S:S + T].cpu().to(torch.float64)
        for got, want, name in ((kg, r["tree_k"][j][sl], "K"), (vg, r["tree_v"][j][sl], "V")):
            err = (got - want).abs()
            assert (err <= ATOL + RTOL * want.abs()).all(), f"tree {name} max err {err.max()}"


def device_setup(w, W_dev, cap_extra=0, seed=0, sampling=False):
    """A Verifier for workload ``w`` with random committed K/V of the
    workload's lengths (std of a real model's cache)."""
    cfg = w.cfg
    caps = [int(s) + len(t[0]) + cap_extra for s, t in zip(w.seq_lens, w.trees)]
    ver = sv.Verifier(cfg, W_dev, caps, max_batch=w.batch, max_tokens=w.n_tokens,
                      sampling=sampling)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    for b, S in enumerate(w.seq_lens):
        k, v = ver.kv.sample_view(b)
        wl.fill_prefix_kv(k, v, int(S), wl.prefix_kv_std(cfg), gen)
    torch.cuda.synchronize()
    return ver


def release(*objs):
    for o in objs:
        del o
    gc.collect()
    torch.cuda.empty_cache()


def shallow(w, layers=2):
    """The same workload on a ``layers``-deep model of the same shape."""
    w.cfg = dataclasses.replace(w.cfg, n_layers=layers)
    return w


def tiny_setup(seed=0, batch=4, chain=4, extra_cap=64, sampling=False, max_tokens=None):
    """The 2-layer workload: bf16-rounded weights, oracle prefill of each
    128-token prompt written into the pool, root = the oracle's greedy token
    after the prompt, chain drafts following the oracle's greedy choice."""
    cfg = wl.TINY
    w = wl.tiny_workload(seed, batch=batch, chain=chain)
    W_cpu = wl.make_weights(cfg, 10 + seed, device="cpu", dtype=torch.bfloat16)
    W_dev = {"tok_embed": W_cpu["tok_embed"].cuda(), "final_norm": W_cpu["final_norm"].cuda(),
             "lm_head": W_cpu["lm_head"].cuda(),
             "layers": [{k: v.cuda() for k, v in lw.items()} for lw in W_cpu["layers"]]}
    caps = [int(s) + extra_cap for s in w.seq_lens]
    ver = sv.Verifier(cfg, W_dev, caps, max_batch=batch, max_tokens=max_tokens or batch * 64,
                      sampling=sampling)
    for b, prompt in enumerate(w.prompts):
        pk, pv, logits = oracle.prefill(cfg, W_cpu, prompt, cache_dtype=torch.bfloat16)
        k, v = ver.kv.sample_view(b)
        k[:, :, :len(prompt)].copy_(pk.cuda())
        v[:, :, :len(prompt)].copy_(pv.cuda())
        w.trees[b][0][0] = int(torch.argmax(logits[-1]))
    torch.cuda.synchronize()
    return cfg, w, W_cpu, W_dev, ver


def oracle_greedy_fn(cfg, W_cpu, ver, ids, lens):
    pk, pv = prefix_for_oracle(ver, ids, lens)

    def fn(trees):
        r = oracle.verify(cfg, W_cpu, pk, pv, lens, trees)
        offs = split_rows(trees)
        g = r["argmax"].tolist()
        return [g[offs[b]:offs[b + 1]] for b in range(len(trees))]

    return fn


def sweep_setup(cfg, W_dev, seed=4000):
    """The launch configuration the strategy-cost sweep times: one pool of the
    256 sweep samples (lognormal committed lengths, room for a 64-node tree
    each) and one verifier sized for 256 samples x 64 nodes; a batch-B cell
    takes the first B samples."""
    lens_all = [int(x) for x in wl.sweep_lengths(seed)]
    caps = [S + max(wl.SWEEP_BUDGETS) for S in lens_all]
    max_b = max(wl.SWEEP_BATCHES)
    ver = sv.Verifier(cfg, W_dev, caps, max_batch=max_b, max_tokens=max_b * max(wl.SWEEP_BUDGETS))
    gen = torch.Generator(device="cuda").manual_seed(seed)
    for b, S in enumerate(lens_all):
        k, v = ver.kv.sample_view(b)
        wl.fill_prefix_kv(k, v, S, wl.prefix_kv_std(cfg), gen)
    torch.cuda.synchronize()
    return ver
