"""Benchmark of the batched tree-verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload early|tail|llama1b]

A step is one verify (target forward over every draft tree, greedy
acceptance) plus the commit (KV compaction) of the whole batch.  Inputs are
synthetic with the shapes of the chosen workload, weights random with the
model's architecture, all resident in HBM before timing starts.  Prints one
JSON line: verified tokens/s as `value`, accepted tokens/s beside it, the
roofline fraction of the dominant kernel (timed with HIP events on its own
stream inside the timed region) and the oracle's throughput on the host cores
over a bounded sample of the same workload.
"""

import argparse
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tree-verify tokens/s & accepted tokens/s, Llama-3-8B shape, 1 MI355X"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
FEW_ROWS_GATE_UP = 4           # gate/up rows up to which the library runs its few-rows kernel


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="early",
                   help="early | tail | llama1b | sweep_b<B>_n<n> (one strategy-cost sweep cell)")
    p.add_argument("--cpu-baseline", type=int, default=1, help="0 skips the oracle timing")
    p.add_argument("--temperature", type=float, default=0.0,
                   help="> 0: speculative-sampling acceptance at this temperature (draft rows "
                        "0.7 p + 0.3 random, seeded uniforms); 0: greedy")
    p.add_argument("--eos", type=int, default=-1, help="end-of-sequence token (-1: none)")
    p.add_argument("--seed", type=int, default=None)
    p.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                   help="only copy BYTES device-to-device 5 times (a reference for the HBM "
                        "byte counters) and exit")
    p.add_argument("--kv-migrate", action="store_true",
                   help="time the migration buffer instead: pack + unpack of 16 samples' K/V "
                        "at the Llama-3-8B shape (lognormal lengths, median 1024)")
    p.add_argument("--trajectory", default=None, metavar="OUT.jsonl",
                   help="run the RLHF generation trajectory (shrinking batch) once per drafting "
                        "strategy (fixed draft token num, or the workload-aware selection) and "
                        "write one JSON line per step to OUT.jsonl")
    p.add_argument("--sweep", default=None, metavar="OUT.jsonl",
                   help="run the strategy-cost sweep (batch x tree budget) and write one JSON "
                        "line per cell to OUT.jsonl")
    return p.parse_args()


def run_sweep(args, out_path):
    """Strategy-cost surface of the verify step: Llama-3-8B shape, batch in
    {1,4,16,64,256} x draft-tree budget n in {1,4,8,16,32,64} (top-n nodes by
    draft logit), one pool of 256 samples with lognormal KV lengths (median
    2048, sigma 0.8, clipped to [128, 16384]); a batch-B cell uses the first B
    samples.  Per cell: verify+commit latency (median over the timed steps),
    verified and accepted tokens/s and the composite roofline fraction."""
    import torch

    import paper_2512_04752_amd as sv
    import workload as wl

    cfg = wl.LLAMA_8B
    lens_all = [int(x) for x in wl.sweep_lengths()]

    W = wl.make_weights(cfg, 4000, device="cuda")
    caps = [S + max(wl.SWEEP_BUDGETS) for S in lens_all]
    max_b = max(wl.SWEEP_BATCHES)
    ver = sv.Verifier(cfg, W, caps, max_batch=max_b, max_tokens=max_b * max(wl.SWEEP_BUDGETS))
    gen = torch.Generator(device="cuda").manual_seed(4000)
    for b, S in enumerate(lens_all):
        k, v = ver.kv.sample_view(b)
        wl.fill_prefix_kv(k, v, S, wl.prefix_kv_std(cfg), gen)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    rows = []
    with open(out_path, "w") as f:
        for B in wl.SWEEP_BATCHES:
            for n in wl.SWEEP_BUDGETS:
                w = wl.sweep_workload(B, n)
                ids, lens = list(range(B)), [int(x) for x in w.seq_lens]

                def greedy_fn(trees):
                    N = sum(len(t[0]) for t in trees)
                    dbg = ver.debug_buffers(N, logits=False)
                    ver.verify(ids, trees, lens, debug=dbg)
                    g = dbg["argmax"].cpu().tolist()
                    res, off = [], 0
                    for t in trees:
                        res.append(g[off:off + len(t[0])])
                        off += len(t[0])
                    return res

                wl.follow_greedy(w.trees, w.branches, w.p_follow, greedy_fn,
                                 np.random.default_rng(4000 + n))
                flat = sv.flatten_trees(w.trees)
                for _ in range(args.warmup):
                    ver.verify(ids, None, lens, flat=flat, stream=stream)
                    ver.commit(ids, lens, stream=stream)
                torch.cuda.synchronize()
                # Median of the per-step times (HIP events on the launch stream),
                # so that one slow step does not move a cell of the cost surface.
                evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                       for _ in range(args.steps)]
                for e0, e1 in evs:
                    e0.record(stream)
                    ver.verify(ids, None, lens, flat=flat, stream=stream)
                    ver.commit(ids, lens, stream=stream)
                    e1.record(stream)
                torch.cuda.synchronize()
                ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in evs]))
                acc = int(ver.accepted_len[:B].sum().item()) + B
                N = w.n_tokens
                kv = sum(S + len(t[0]) for S, t in zip(lens, w.trees))
                t_roof = max(2.0 * N * cfg.gemm_params() / (PEAK_BF16_TFLOPS * 1e12),
                             2.0 * cfg.gemm_params() / (PEAK_HBM_GBS * 1e9)) + \
                    kv * cfg.kv_bytes_per_token() / (PEAK_HBM_GBS * 1e9)
                row = {"batch": B, "budget": n, "tokens": N, "kv_tokens": kv,
                       "ms_per_step": round(ms, 4), "verified_tokens_per_s": round(N / ms * 1e3, 1),
                       "accepted_tokens_per_s": round(acc / ms * 1e3, 1),
                       "accepted_per_sample": round(acc / B, 3),
                       "t_roof_ms": round(t_roof * 1e3, 4), "roofline_frac": round(t_roof * 1e3 / ms, 4)}
                rows.append(row)
                f.write(json.dumps(row) + "\n")
                f.flush()
                print(json.dumps(row), file=sys.stderr, flush=True)
    return rows


def run_kv_migrate(args):
    """Sample migration's KV transfer (paper Section 6.2, phases 1 and 3) at the
    Llama-3-8B shape: 16 samples with lognormal committed lengths (median 1024,
    sigma 0.8, clipped to [128, 8192], the early-generation distribution) are
    packed from a source pool into one contiguous buffer and unpacked into a
    destination pool.  Each kernel moves every byte twice (read + write); the
    bound is HBM bandwidth."""
    import torch

    import paper_2512_04752_amd as sv
    import workload as wl

    cfg = wl.LLAMA_8B
    rng = np.random.default_rng(6000)
    lens = [int(x) for x in np.clip(np.round(rng.lognormal(np.log(1024), 0.8, 16)), 128, 8192)]
    src = sv.KVPool(cfg, lens)
    dst = sv.KVPool(cfg, [max(lens) + 64] * 16)
    src.buf.fill_(1)
    ids = list(range(16))
    dids = ids[::-1]
    begin, end = [0] * 16, lens
    nbytes = sv.spec_kv_transfer_bytes(src, begin, end)
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        sv.spec_kv_pack(src, ids, begin, end, buf, stream=stream)
        sv.spec_kv_unpack(dst, dids, begin, end, buf, stream=stream)
    torch.cuda.synchronize()
    res = {}
    for name, fn in (("pack", lambda: sv.spec_kv_pack(src, ids, begin, end, buf, stream=stream)),
                     ("unpack", lambda: sv.spec_kv_unpack(dst, dids, begin, end, buf,
                                                          stream=stream))):
        sv.spec_profile_begin("transfer", args.steps + 1)
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        ms, n = sv.spec_profile_end()
        avg = ms / max(n, 1)
        gbs = 2 * nbytes / (avg / 1e3) / 1e9
        res[name] = {"avg_launch_ms": round(avg, 4), "launches": n, "achieved": round(gbs, 1),
                     "frac": round(gbs / PEAK_HBM_GBS, 4)}
    return {"metric": "KV transfer GB/s (read + write), sample migration phases 1 and 3",
            "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "config": {"workload": "Llama-3-8B shape, 16 samples, KV lengths lognormal(median "
                                   "1024, sigma 0.8) in [128, 8192]", "tokens": int(sum(lens)),
                       "buffer_bytes": int(nbytes)},
            "dtype": "bf16 (bytes copied)", "roofline": {"bound": "hbm", "peak": PEAK_HBM_GBS,
                                                          "unit": "GB/s", "pack": res["pack"],
                                                          "unpack": res["unpack"]}}


def run_trajectory(args, out_path):
    """Generation stage of one RLHF iteration on one instance, with each
    drafting strategy (paper Sections 5 and 7.3): 128 samples at the
    Llama-3-8B shape, prompts with the early-generation length distribution
    (lognormal, median 1024, sigma 0.8, clipped to [128, 8192]) and response
    lengths lognormal(median 378, sigma 0.784) clipped to [1, 2048] (the
    paper's LMSYS response statistics: median 378, 95th percentile 1373).
    A sample leaves the batch once it has generated its response.

    Every step: each live sample gets a candidate draft tree (top-64 nodes by
    draft logit of a depth-8, 4-ary tree with Dirichlet(1) sibling scores;
    node weight w = F(dl) with a linear F of slope 1); the strategy picks the
    draft token num n (fixed, or spec_select_draft_count with the cost model
    fitted on this GPU); the top-n nodes are verified by spec_verify (real
    kernels, random draft tokens); the accepted branch is then drawn from the
    same acceptance model the selector assumes (child c of an accepted node u
    is accepted with probability w(c) / w(u), siblings exclusive), and
    spec_kv_commit compacts it.  Time per step: host selection and tree
    building + verify + commit, synchronised."""
    import torch

    import paper_2512_04752_amd as sv
    import workload as wl

    cfg = wl.LLAMA_8B
    B0 = 128
    rng = np.random.default_rng(7000)
    prompts = [int(x) for x in wl.lognormal_lengths(rng, B0, 1024, 0.8, 128, 8192)]
    resp = [int(x) for x in np.clip(np.round(rng.lognormal(np.log(378), 0.784, B0)), 1, 2048)]
    pool_trees = []
    for _ in range(512):
        par, dl = wl.draft_logit_tree(rng, 64)
        pool_trees.append((par, [float(x) for x in dl]))
    caps = [p + r + 80 for p, r in zip(prompts, resp)]
    W = wl.make_weights(cfg, 7000, device="cuda")
    ver = sv.Verifier(cfg, W, caps, max_batch=B0, max_tokens=B0 * 64)
    data_dir = os.path.join(ROOT, "paper_2512_04752_amd", "data")
    coeffs = json.load(open(os.path.join(data_dir, "verify_cost_model__llama8b_mi355x.json")))
    model = sv.CostModel.from_dict(coeffs)
    stream = torch.cuda.current_stream()
    strategies = [("fixed", n) for n in (1, 4, 8, 16, 32)] + [("adaptive", 64)]
    summary = []
    with open(out_path, "w") as fout:
        for kind, nmax in strategies:
            gen = torch.Generator(device="cuda").manual_seed(7000)
            for b, S in enumerate(prompts):
                k, v = ver.kv.sample_view(b)
                wl.fill_prefix_kv(k, v, S, wl.prefix_kv_std(cfg), gen)
            torch.cuda.synchronize()
            r_step = np.random.default_rng(7001)
            live = list(range(B0))
            S_len = list(prompts)
            done = [0] * B0
            steps, t_total, t_gpu, tokens, n_sum = 0, 0.0, 0.0, 0, 0
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            while live:
                t0 = time.perf_counter()
                picks = r_step.integers(0, len(pool_trees), len(live))
                trees = [pool_trees[i] for i in picks]
                offs = np.zeros(len(live) + 1, dtype=np.int32)
                offs[1:] = np.cumsum([len(t[0]) for t in trees])
                pars = np.fromiter((x for t in trees for x in t[0]), dtype=np.int32)
                ws = np.fromiter((x for t in trees for x in t[1]), dtype=np.float32)
                lens = [S_len[b] for b in live]
                n_sel, order, _ = sv.spec_select_draft_count(model, lens, offs, pars, ws,
                                                             nmax if kind == "adaptive" else nmax,
                                                             patience=2)
                n = n_sel if kind == "adaptive" else nmax
                vtrees, vweights = [], []
                for j, (par, w) in enumerate(trees):
                    ids = [int(x) for x in order[j, :n] if x >= 0]
                    pos = {u: k for k, u in enumerate(ids)}
                    vpar = [-1] + [pos[par[u]] for u in ids[1:]]
                    vtrees.append((wl.random_tokens(r_step, len(ids), cfg.vocab), vpar))
                    vweights.append([w[u] for u in ids])
                # acceptance drawn from the weights (the selector's own model)
                acc_len = np.zeros(len(live), dtype=np.int32)
                acc_nodes = np.full((len(live), sv.SPEC_MAX_TREE), -1, dtype=np.int32)
                for j, ((tok, vpar), w) in enumerate(zip(vtrees, vweights)):
                    kids = [[] for _ in vpar]
                    for k in range(1, len(vpar)):
                        kids[vpar[k]].append(k)
                    u, path = 0, [0]
                    while kids[u]:
                        x = r_step.random() * w[u]
                        nxt = -1
                        for c in kids[u]:
                            if x < w[c]:
                                nxt = c
                                break
                            x -= w[c]
                        if nxt < 0:
                            break
                        u = nxt
                        path.append(u)
                    acc_len[j] = len(path) - 1
                    acc_nodes[j, :len(path)] = path
                ev0.record(stream)
                ver.verify(live, vtrees, lens, stream=stream)
                ver.accepted_len[:len(live)].copy_(torch.from_numpy(acc_len), non_blocking=False)
                ver.accepted_nodes[:len(live)].copy_(torch.from_numpy(acc_nodes), non_blocking=False)
                ver.commit(live, lens, stream=stream)
                ev1.record(stream)
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                dt_gpu = ev0.elapsed_time(ev1)
                gained = 0
                still = []
                for j, b in enumerate(live):
                    g = int(acc_len[j]) + 1
                    S_len[b] += g
                    done[b] += g
                    gained += g
                    if done[b] < resp[b]:
                        still.append(b)
                fout.write(json.dumps({"strategy": f"{kind}_{nmax}", "step": steps, "batch": len(live),
                                       "n": int(n), "ms": round((t1 - t0) * 1e3, 3),
                                       "gpu_ms": round(dt_gpu, 3), "tokens": gained}) + "\n")
                steps += 1
                t_total += t1 - t0
                t_gpu += dt_gpu / 1e3
                tokens += gained
                n_sum += n
                live = still
            row = {"strategy": kind if kind == "adaptive" else f"fixed n={nmax}", "steps": steps,
                   "tokens": tokens, "seconds": round(t_total, 3),
                   "tokens_per_s": round(tokens / t_total, 1),
                   "gpu_tokens_per_s": round(tokens / t_gpu, 1), "mean_n": round(n_sum / steps, 2)}
            summary.append(row)
            print(json.dumps(row), file=sys.stderr, flush=True)
    hits, misses = model.stats()
    return {"metric": "RLHF generation trajectory: generated tokens/s per drafting strategy",
            "unit": "tokens/s", "n_gpus": 1,
            "config": {"workload": "Llama-3-8B shape, 128 samples, prompts lognormal(1024, 0.8), "
                                   "responses lognormal(378, 0.784) in [1, 2048], top-64 "
                                   "draft-logit candidate trees, acceptance drawn from w = dl"},
            "strategies": summary, "cost_model_cache": {"hits": hits, "misses": misses},
            "out": out_path}


def recorded_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    copy-calibrated rocprofv3 counter summary, or None when there is none or
    the kernel's source has changed since the counters were taken."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic__*.md")):
        for line in open(path):
            f = line.split()
            if len(f) != 6 or f[0] != "traffic" or f[1] != workload or f[2] != kernel:
                continue
            kv = dict(x.split("=", 1) for x in f[3:])
            src = os.path.join(ROOT, kv["source"])
            if os.path.exists(src) and hashlib.sha1(open(src, "rb").read()).hexdigest() == kv["sha1"]:
                return int(float(kv["bytes_per_launch"]))
    return None


def attention_kernels(cfg, w):
    """Kernels one attention launch runs for this workload's tree sizes."""
    G = cfg.n_heads // cfg.n_kv_heads
    tiles = [(len(t[0]) * G + 31) // 32 for t in w.trees]
    names = []
    if min(tiles) == 1:
        names.append(f"tree_attention_kernel<{cfg.head_dim}>")
    if any(1 < t <= 4 for t in tiles):
        names.append(f"tree_attention_wide_kernel<{cfg.head_dim},4>")
    if max(tiles) > 4:
        names.append(f"tree_attention_wide_kernel<{cfg.head_dim},8>")
    return names


def make_workload(name, seed):
    import workload as wl
    m = re.fullmatch(r"sweep_b(\d+)_n(\d+)", name)
    if m:
        return wl.sweep_workload(int(m.group(1)), int(m.group(2)), *(() if seed is None else (seed,)))
    make = {"early": wl.early_workload, "tail": wl.tail_workload, "llama1b": wl.llama1b_workload}
    if name not in make:
        raise SystemExit(f"unknown workload {name!r}")
    return make[name]() if seed is None else make[name](seed)


def describe(name, w):
    if name.startswith("sweep"):
        return (f"Llama-3-8B-shape verify, sweep cell: batch {w.batch}, top-{len(w.trees[0][0])} "
                "draft-logit trees, KV lengths lognormal(median 2048, sigma 0.8) in [128, 16384]")
    if name == "early":
        return ("Llama-3-8B-shape verify, early generation: batch 128, 8-node draft trees "
                "(4 levels, width <= 3), KV lengths lognormal(median 1024, sigma 0.8) in [128, 8192]")
    if name == "tail":
        return ("Llama-3-8B-shape verify, long tail: batch 4, 64-node draft trees (8 levels, "
                "<= 4 children), KV lengths U[16384, 32768]")
    return ("Llama-3.2-1B-shape verify: batch 32, 15-node binary trees, KV lengths U[512, 2048]")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch

    import paper_2512_04752_amd as sv
    import workload as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        src = torch.ones(args.copy_calibration, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.copy_calibration, "copies": 5}), flush=True)
        return
    if args.kv_migrate:
        print(json.dumps(run_kv_migrate(args)), flush=True)
        return
    if args.trajectory:
        print(json.dumps(run_trajectory(args, args.trajectory)), flush=True)
        return
    if args.sweep:
        rows = run_sweep(args, args.sweep)
        best = max(rows, key=lambda r: r["accepted_tokens_per_s"])
        print(json.dumps({"metric": METRIC + " (strategy-cost sweep)", "cells": len(rows),
                          "best_accepted_tokens_per_s": best["accepted_tokens_per_s"],
                          "best_cell": {"batch": best["batch"], "budget": best["budget"]},
                          "out": args.sweep}), flush=True)
        return
    w = make_workload(args.workload, args.seed)
    cfg = w.cfg
    plain_trees = [(list(t[0]), list(t[1])) for t in w.trees]   # before greedy steering

    t_setup = time.time()
    W = wl.make_weights(cfg, w.seed, device="cuda")
    caps = [int(s) + len(t[0]) for s, t in zip(w.seq_lens, w.trees)]
    sampled = args.temperature > 0 or args.eos >= 0
    ver = sv.Verifier(cfg, W, caps, max_batch=w.batch, max_tokens=w.n_tokens,
                      sampling=args.temperature > 0)
    gen = torch.Generator(device="cuda").manual_seed(w.seed)
    for b, S in enumerate(w.seq_lens):
        k, v = ver.kv.sample_view(b)
        wl.fill_prefix_kv(k, v, int(S), wl.prefix_kv_std(cfg), gen)
    ids = list(range(w.batch))
    lens = [int(s) for s in w.seq_lens]

    # Draft trees whose designated branch follows the target's greedy choice
    # (p = 0.7 per level), built with untimed verify calls.
    def greedy_fn(trees):
        n = sum(len(t[0]) for t in trees)
        dbg = ver.debug_buffers(n, logits=False)
        ver.verify(ids, trees, lens, debug=dbg)
        g = dbg["argmax"].cpu().tolist()
        out, off = [], 0
        for t in trees:
            out.append(g[off:off + len(t[0])])
            off += len(t[0])
        return out

    wl.follow_greedy(w.trees, w.branches, w.p_follow, greedy_fn, np.random.default_rng(w.seed))
    flat = sv.flatten_trees(w.trees)
    q_rows = uniforms = None
    if args.temperature > 0:
        # draft rows: 0.7 of the target's own distribution plus 0.3 of a
        # random one, from an untimed verify's logits; seeded uniforms
        dbg = ver.debug_buffers(w.n_tokens, logits=True)
        ver.verify(ids, w.trees, lens, debug=dbg)
        q_rows = torch.empty(w.n_tokens, cfg.vocab, dtype=torch.float32, device="cuda")
        for r0 in range(0, w.n_tokens, 256):
            z = dbg["logits"][r0:r0 + 256].double()
            r = torch.softmax(torch.randn(z.shape, generator=gen, device="cuda",
                                          dtype=torch.float64) * 2.0, dim=1)
            q = 0.7 * torch.softmax(z / args.temperature, dim=1) + 0.3 * r
            q_rows[r0:r0 + 256] = (q / q.sum(dim=1, keepdim=True)).float()
        del dbg
        u = np.random.default_rng(w.seed + 1).uniform(0, 1, (w.n_tokens, 2)).astype(np.float32)
        uniforms = torch.from_numpy(np.minimum(u, np.float32(1 - 2 ** -24))).cuda()
    torch.cuda.synchronize()
    setup_s = time.time() - t_setup

    stream = torch.cuda.current_stream()

    def step():
        if sampled:
            ver.verify_sampled(ids, None, lens, args.temperature, args.eos, q_rows, uniforms,
                               flat=flat, stream=stream)
        else:
            ver.verify(ids, None, lens, flat=flat, stream=stream)
        ver.commit(ids, lens, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Timed region: K steps between synchronisations, nothing else enqueued.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps

    # Dominant kernel: every launch bracketed by HIP events on its own stream
    # over a second timed pass of the same K steps (kept apart so that the
    # event records do not enter the step time above).
    dominant = "attention" if args.workload == "tail" else "gemm_gate_up"
    sv.spec_profile_begin(dominant, args.steps * cfg.n_layers + 8)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    dom_ms, dom_launches = sv.spec_profile_end()
    ms_per_step_events = (t3 - t2) * 1e3 / args.steps

    acc = ver.accepted_len[:w.batch].cpu()
    accepted = int(acc.sum().item()) + w.batch          # + the bonus token per sample
    n_tok = w.n_tokens
    value = n_tok / (ms_per_step / 1e3)
    acc_rate = accepted / (ms_per_step / 1e3)

    # Per-kernel-class time of one step, measured in separate untimed steps.
    breakdown = {}
    for kc in sv.binding.KERNEL_CLASS:
        sv.spec_profile_begin(kc, 4 * cfg.n_layers + 8)
        step()
        torch.cuda.synchronize()
        ms, n = sv.spec_profile_end()
        breakdown[kc] = round(ms, 4)

    # Roofline of the dominant kernel: algorithmic work of one launch.
    H, F, d = cfg.hidden, cfg.ffn, cfg.head_dim
    avg_ms = dom_ms / max(dom_launches, 1)
    gu_flops = 2.0 * n_tok * (2 * F) * H
    gu_bytes = 2 * F * H * 2 + n_tok * (H + F) * 2     # weights + activations in + out
    if dominant == "gemm_gate_up" and gu_flops / (PEAK_BF16_TFLOPS * 1e12) >= \
            gu_bytes / (PEAK_HBM_GBS * 1e9):
        achieved = gu_flops / (avg_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": recorded_traffic(args.workload, "gemm_bf16_kernel<EPI_GATE_UP>"),
                "kernel": "gemm_bf16_kernel<EPI_GATE_UP>",
                "work_per_launch": f"2*{n_tok}*{2 * F}*{H} flop"}
    elif dominant == "gemm_gate_up":
        achieved = gu_bytes / (avg_ms / 1e3) / 1e9
        # up to FEW_ROWS_GATE_UP rows the product runs the few-rows kernel
        # (no K split leaves the work-group), otherwise the tile kernel
        gu_kern = ("skinny_gemm_kernel<EPI_GATE_UP>" if n_tok <= FEW_ROWS_GATE_UP
                   else "gemm_bf16_kernel<EPI_GATE_UP> (+ split-K reduce)")
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": recorded_traffic(args.workload, "gemm_bf16_kernel<EPI_GATE_UP>"),
                "kernel": gu_kern,
                "work_per_launch": f"{gu_bytes} bytes (gate and up weights once, rows in and out)"}
    else:
        work = attention_work(cfg, w)
        achieved = work / (avg_ms / 1e3) / 1e9
        kern = " + ".join(attention_kernels(cfg, w) + [f"attention_combine_kernel<{d}>"])
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": recorded_traffic(args.workload, kern.replace(" ", "")),
                "kernel": kern,
                "work_per_launch": f"{work} bytes (K/V of every key once, q in, o out)"}
    roof["avg_launch_ms"] = round(avg_ms, 5)
    roof["launches"] = dom_launches
    roof["timed_pass_ms_per_step"] = round(ms_per_step_events, 4)

    # Composite roofline of the whole step.
    gemm_flops = 2.0 * n_tok * cfg.gemm_params()
    attn_bytes = sum((int(S) + len(t[0])) for S, t in zip(w.seq_lens, w.trees)) * \
        cfg.kv_bytes_per_token()
    weight_bytes = 2.0 * cfg.gemm_params()
    t_roof = max(gemm_flops / (PEAK_BF16_TFLOPS * 1e12), weight_bytes / (PEAK_HBM_GBS * 1e9)) + \
        attn_bytes / (PEAK_HBM_GBS * 1e9)

    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (random weights of the named shape, synthetic KV and draft trees)",
        "config": {"workload": describe(args.workload, w), "model": "llama-3-8b-shape"
                   if cfg.hidden == 4096 else "llama-3.2-1b-shape",
                   "batch": w.batch, "tokens_per_step": n_tok,
                   "kv_tokens": int(sum(lens)), "parallelism": "none (1 GPU)"},
        "accepted_tokens_per_s": round(acc_rate, 1),
        "accepted_per_sample_per_step": round(accepted / w.batch, 3),
        "roofline": roof,
        "step_roofline": {"t_roof_ms": round(t_roof * 1e3, 4),
                          "frac": round(t_roof * 1e3 / ms_per_step, 4)},
        "breakdown_ms_per_step": breakdown,
        "setup_s": round(setup_s, 1),
    }
    if sampled:
        result["config"]["acceptance"] = (f"speculative sampling, T = {args.temperature}"
                                          if args.temperature > 0 else "greedy") + \
            (f", EOS token {args.eos}" if args.eos >= 0 else "")
    if args.temperature > 0:
        result["sampled_accept"] = sampled_accept_roofline(cfg, w, ver, breakdown["accept"],
                                                           ms_per_step)
    result["attention"] = attention_roofline(cfg, w, breakdown["attention"])
    result["compaction"] = compaction_roofline(cfg, w, ver, breakdown["commit"])

    if args.cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, W, ver, w, plain_trees, lens, n_tok,
                                              ms_per_step)
    print(json.dumps(result), flush=True)


def attention_work(cfg, w):
    """Algorithmic bytes of one layer's tree attention: the K and V rows of
    every committed and tree key once, the queries in and the outputs out."""
    d = cfg.head_dim
    kv_bytes = sum((int(S) + len(t[0])) for S, t in zip(w.seq_lens, w.trees)) * \
        cfg.n_kv_heads * d * 2 * 2
    qo_bytes = w.n_tokens * cfg.n_heads * d * 2 * 2
    return kv_bytes + qo_bytes


def attention_roofline(cfg, w, attn_ms):
    """Tree attention of one step (every layer, split-KV merge included)
    against HBM bandwidth, whichever kernel class dominates the step."""
    alg = attention_work(cfg, w) * cfg.n_layers
    gbs = alg / (attn_ms / 1e3) / 1e9 if attn_ms > 0 else 0.0
    return {"bound": "hbm", "bytes_per_step": alg, "ms_per_step": attn_ms,
            "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 4),
            "kernel": " + ".join(attention_kernels(cfg, w) +
                                 [f"attention_combine_kernel<{cfg.head_dim}>"])}


def compaction_roofline(cfg, w, ver, commit_ms):
    """The KV compaction of one commit against HBM bandwidth.  Algorithmic
    bytes: every accepted node not already at its final slot (node index !=
    depth) has its K and V rows of every layer and KV head read once and
    written once."""
    acc = ver.accepted_len[:w.batch].cpu().tolist()
    nodes = ver.accepted_nodes[:w.batch].cpu().tolist()
    moved = sum(1 for b in range(w.batch) for dd in range(1, acc[b] + 1) if nodes[b][dd] != dd)
    row_bytes = cfg.n_layers * 2 * cfg.n_kv_heads * cfg.head_dim * 2
    alg = 2 * moved * row_bytes
    gbs = alg / (commit_ms / 1e3) / 1e9 if commit_ms > 0 else 0.0
    return {"bound": "hbm", "moved_rows": moved, "bytes_per_commit": alg,
            "ms_per_commit": commit_ms, "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4), "kernel": "compact_kernel"}


def sampled_accept_roofline(cfg, w, ver, accept_ms, ms_per_step):
    """The sampled-acceptance kernel against HBM bandwidth.  Algorithmic
    bytes: each node on a sample's walk reads its fp32 logit row, and its
    fp32 draft row when it has children to try."""
    acc = ver.accepted_len[:w.batch].cpu().tolist()
    nodes = ver.accepted_nodes[:w.batch].cpu().tolist()
    rows = 0
    for b, (toks, pars) in enumerate(w.trees):
        for u in nodes[b][:acc[b] + 1]:
            rows += 2 if any(p == u for p in pars[1:]) else 1
    alg = rows * cfg.vocab * 4
    gbs = alg / (accept_ms / 1e3) / 1e9
    return {"kernel": "node_decide_kernel<1024> + sample_walk_kernel<1024>",
            "avg_launch_ms": round(accept_ms, 5),
            "share_of_step": round(accept_ms / ms_per_step, 4), "bound": "hbm",
            "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 4),
            "work_per_launch": f"{alg} bytes ({rows} vocabulary rows of fp32)"}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, W, ver, w, plain_trees, lens, n_tok, ms_per_step):
    """The oracle, untuned, on the host cores over a bounded sample: one
    batched verify call over 4 samples (more for small trees, so that the
    sample holds at least 64 tree nodes) of the workload taken at
    evenly spaced quantiles of its committed lengths (so the sample follows
    the workload's length distribution), with their unsteered draft trees.
    A second call on the same trees with empty prefixes separates the cost
    that grows with the tree nodes (matrix products) from the cost that grows
    with nodes x committed length (attention), which gives an extrapolation
    to the whole batch: c_node * N + c_attn * sum_b T_b * S_b."""
    import torch

    import oracle

    threads = len(os.sched_getaffinity(0))
    torch.set_num_threads(threads)
    Wc = {"tok_embed": W["tok_embed"].cpu(), "final_norm": W["final_norm"].cpu(),
          "lm_head": W["lm_head"].cpu(),
          "layers": [{k: v.cpu() for k, v in lw.items()} for lw in W["layers"]]}
    order = np.argsort(np.asarray(lens), kind="stable")
    k = min(w.batch, max(4, -(-64 * w.batch // n_tok)))
    pick = sorted({int(order[int((i + 0.5) * len(order) / k)]) for i in range(k)})
    pk = [ver.kv.sample_view(b)[0][:, :, :lens[b]].cpu() for b in pick]
    pv = [ver.kv.sample_view(b)[1][:, :, :lens[b]].cpu() for b in pick]
    trees = [plain_trees[b] for b in pick]
    t0 = time.perf_counter()
    oracle.verify(cfg, Wc, pk, pv, [lens[b] for b in pick], trees)
    t_full = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.verify(cfg, Wc, None, None, [0] * len(pick), trees)
    t_nodes = time.perf_counter() - t0
    toks = sum(len(t[0]) for t in trees)
    tk_sample = sum(len(plain_trees[b][0]) * lens[b] for b in pick)
    tk_full = sum(len(t[0]) * S for t, S in zip(plain_trees, lens))
    c_node = t_nodes / toks
    c_attn = max(t_full - t_nodes, 0.0) / max(tk_sample, 1)
    t_batch = c_node * n_tok + c_attn * tk_full
    return {"value": round(toks / t_full, 4), "unit": "tokens/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{len(pick)} of the workload's {w.batch} samples at evenly spaced quantiles "
                      f"of its committed lengths (KV {[lens[b] for b in pick]}, mean "
                      f"{np.mean([lens[b] for b in pick]):.0f} vs the workload's "
                      f"{np.mean(lens):.0f}), {toks} tree nodes, one batched call of the "
                      f"float64 torch-CPU oracle: {t_full:.1f} s ({t_nodes:.1f} s with empty "
                      f"prefixes)",
            "measured_s": round(t_full, 2),
            "extrapolated": {"s_per_step": round(t_batch, 1),
                             "tokens_per_s": round(n_tok / t_batch, 4),
                             "method": "extrapolated to the whole batch: per-node cost x N + "
                                       "per-(T_b x S_b) attention cost x sum T_b S_b"}}


if __name__ == "__main__":
    main()
