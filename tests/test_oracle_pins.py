"""Pins of the oracle against facts that do not come from the oracle itself.

* hand-derived closed forms (RMSNorm, rotary embedding, softmax weights,
  tree depths and ancestor sets);
* brute force: acceptance by enumerating every branch of the tree;
* an independent decoder (Hugging Face Llama, float64): every node's logits
  must equal those of its branch decoded on its own after the prompt, and
  chain drafts with greedy acceptance must reproduce plain greedy decoding
  token for token (the lossless property of speculative decoding,
  Section 2.2);
* special cases: a one-node tree is one autoregressive step, a star tree is
  a set of independent one-token continuations, nkv = nq is ordinary
  multi-head attention, relabelling the nodes permutes the results;
* the bf16-operand mode (the ideal bf16 computation that sets the tolerance
  of full-depth GPU comparisons) against the same independent decoder with
  every bf16 storage point rounded by hooks on its own modules: equal to
  rounding order, while leaving out any one rounding point moves the logits
  by more than 1e-3.

All CPU; no GPU needed.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import workload as wl
from tests.hf_ref import STORAGE_POINTS, bf16_storage, hf_greedy, hf_logits, hf_model, hf_model_f64

PIN = wl.ModelConfig(n_layers=2, hidden=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn=128,
                     vocab=97, rope_theta=1e4, rms_eps=1e-5)
PIN_MHA = wl.ModelConfig(n_layers=2, hidden=64, n_heads=4, n_kv_heads=4, head_dim=16, ffn=128,
                         vocab=97, rope_theta=1e4, rms_eps=1e-5)


def pin_weights(cfg, seed, std=0.1):
    """float64 weights with std ``std`` and random (non-unit) norm gains, so
    that a dropped gain or a mis-scaled term changes the logits."""
    W = wl.make_weights(cfg, seed, dtype=torch.float64)
    g = torch.Generator().manual_seed(seed + 17)

    def fix(name, t):
        if name.endswith("norm"):
            return 1.0 + 0.3 * torch.randn(t.shape, generator=g, dtype=torch.float64)
        return t * (std / wl.WEIGHT_STD)

    for lw in W["layers"]:
        for k in list(lw):
            lw[k] = fix(k, lw[k])
    W["tok_embed"] = fix("tok_embed", W["tok_embed"])
    W["lm_head"] = fix("lm_head", W["lm_head"])
    W["final_norm"] = fix("final_norm", W["final_norm"])
    return W


def branch_tokens(tokens, parents, node):
    out = []
    while node != -1:
        out.append(tokens[node])
        node = parents[node] if node != 0 else -1
    return out[::-1]


def run_verify(cfg, W, prompt, tree):
    pk, pv, _ = oracle.prefill(cfg, W, prompt, cache_dtype=torch.float64)
    return oracle.verify(cfg, W, [pk], [pv], [len(prompt)], [tree])


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------

def test_tree_metadata_hand_example():
    parents = [-1, 0, 0, 1, 1, 2, 5]
    depth, anc = oracle.tree_metadata(parents)
    assert depth.tolist() == [0, 1, 1, 2, 2, 2, 3]
    assert anc[6].nonzero().flatten().tolist() == [0, 2, 5, 6]
    assert anc[4].nonzero().flatten().tolist() == [0, 1, 4]
    assert anc[0].nonzero().flatten().tolist() == [0]
    with pytest.raises(ValueError):
        oracle.tree_metadata([-1, 1])
    with pytest.raises(ValueError):
        oracle.tree_metadata([0, -1])


def test_rms_norm_closed_form():
    x = torch.tensor([[3.0, 4.0]], dtype=torch.float64)
    g = torch.tensor([2.0, -1.0], dtype=torch.float64)
    y = oracle.rms_norm(x, g, 0.0)
    # mean square 12.5; 3/sqrt(12.5) = 0.848528137..., 4/sqrt(12.5) = 1.131370849...
    assert torch.allclose(y, torch.tensor([[2 * 0.8485281374238570, -1.1313708498984762]],
                                          dtype=torch.float64), rtol=0, atol=1e-15)
    y = oracle.rms_norm(x, torch.ones(2, dtype=torch.float64), 0.5)
    assert abs(float(y[0, 0]) - 3 / math.sqrt(13.0)) < 1e-15


def test_rope_closed_form():
    # d = 4, theta = 100: frequencies 1 and 0.1.  Pair (x0, x2) turns by p
    # radians, pair (x1, x3) by 0.1 p radians.
    x = torch.tensor([[[1.0, 2.0, 0.0, 0.5]]], dtype=torch.float64)
    for p in (0, 2, 7):
        cos, sin = oracle.rope_cos_sin(torch.tensor([p]), 4, 100.0)
        y = oracle.rope(x, cos, sin)[0, 0]
        a0, b0 = 1.0 * math.cos(p) - 0.0 * math.sin(p), 0.0 * math.cos(p) + 1.0 * math.sin(p)
        w = 0.1 * p
        a1, b1 = 2.0 * math.cos(w) - 0.5 * math.sin(w), 0.5 * math.cos(w) + 2.0 * math.sin(w)
        assert torch.allclose(y, torch.tensor([a0, a1, b0, b1], dtype=torch.float64), atol=1e-14)


def test_rope_relative_position():
    g = torch.Generator().manual_seed(3)
    q = torch.randn(1, 1, 16, generator=g, dtype=torch.float64)
    k = torch.randn(1, 1, 16, generator=g, dtype=torch.float64)

    def dot(m, n):
        cq, sq = oracle.rope_cos_sin(torch.tensor([m]), 16, 1e4)
        ck, sk = oracle.rope_cos_sin(torch.tensor([n]), 16, 1e4)
        return float((oracle.rope(q, cq, sq) * oracle.rope(k, ck, sk)).sum())

    assert abs(dot(5, 2) - dot(105, 102)) < 1e-12
    assert abs(dot(0, 0) - float((q * k).sum())) < 1e-12


def test_attention_softmax_weights():
    # one query, two visible keys plus one masked key
    q = torch.tensor([[[1.0, 0.0]]], dtype=torch.float64)            # [T=1, nq=1, d=2]
    k = torch.tensor([[[2.0, 0.0], [0.0, 1.0], [9.0, 9.0]]], dtype=torch.float64)
    v = torch.tensor([[[1.0, 0.0], [0.0, 1.0], [5.0, 5.0]]], dtype=torch.float64)
    vis = torch.tensor([[True, True, False]])
    o = oracle.attention(q, k, v, vis, 1)
    s1, s2 = 2.0 / math.sqrt(2), 0.0
    w1 = math.exp(s1) / (math.exp(s1) + math.exp(s2))
    assert torch.allclose(o[0, 0], torch.tensor([w1, 1 - w1], dtype=torch.float64), atol=1e-15)


# ---------------------------------------------------------------------------
# acceptance: brute force over every branch
# ---------------------------------------------------------------------------

def brute_accept(tokens, parents, g):
    T = len(tokens)
    best, best_depth = 0, 0
    for i in range(T):
        node, ok, dep = i, True, 0
        while node != 0:
            p = parents[node]
            if tokens[node] != g[p]:
                ok = False
            node, dep = p, dep + 1
        if ok and dep > best_depth:
            best, best_depth = i, dep
    path, node = [], best
    while True:
        path.append(node)
        if node == 0:
            break
        node = parents[node]
    return best_depth, g[best], path[::-1]


@pytest.mark.parametrize("seed", range(40))
def test_acceptance_matches_enumeration(seed):
    rng = np.random.default_rng(seed)
    kind = seed % 4
    if kind == 0:
        T = int(rng.integers(1, 40))
        parents = wl.recursive_tree(rng, T, int(rng.integers(min(T, 4), min(T, 8) + 1)), 4)
    elif kind == 1:
        parents = wl.chain_tree(int(rng.integers(1, 12)))
    elif kind == 2:
        parents = [-1] + [0] * int(rng.integers(0, 10))        # star
    else:
        parents = wl.early_tree(rng)
    T = len(parents)
    alphabet = 2 + seed % 3        # small alphabet: duplicate siblings, many matches
    tokens = [int(t) for t in rng.integers(0, alphabet, T)]
    g = [int(t) for t in rng.integers(0, alphabet, T)]
    assert oracle.greedy_accept(tokens, parents, g) == brute_accept(tokens, parents, g)


def test_acceptance_hand_example():
    parents = [-1, 0, 0, 1, 1, 2, 5]
    tokens = [10, 11, 12, 13, 14, 15, 16]
    # the target predicts 12 after node 0, 15 after node 2, 99 after node 5
    g = [12, 0, 15, 0, 0, 99, 0]
    assert oracle.greedy_accept(tokens, parents, g) == (2, 99, [0, 2, 5])
    # nothing accepted: next token is the prediction after the root
    assert oracle.greedy_accept(tokens, parents, [7] * 7) == (0, 7, [0])


# ---------------------------------------------------------------------------
# the independent decoder
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def pin_setup():
    W = pin_weights(PIN, 11)
    return W, hf_model(PIN, W)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_node_logits_equal_branch_decoding(pin_setup, seed):
    W, model = pin_setup
    rng = np.random.default_rng(100 + seed)
    prompt = wl.random_tokens(rng, 9, PIN.vocab)
    parents = wl.recursive_tree(rng, 20, 6, 3)
    tokens = wl.random_tokens(rng, len(parents), PIN.vocab)
    r = run_verify(PIN, W, prompt, (tokens, parents))
    for i in range(len(parents)):
        ref = hf_logits(model, prompt + branch_tokens(tokens, parents, i))[-1]
        err = (r["logits"][i] - ref).abs().max().item()
        assert err < 1e-5 * max(1.0, ref.abs().max().item()), (i, err)
    depth, _ = oracle.tree_metadata(parents)
    assert r["pos"].tolist() == (len(prompt) + depth).tolist()


def test_prefill_matches_causal_decoding(pin_setup):
    W, model = pin_setup
    rng = np.random.default_rng(5)
    prompt = wl.random_tokens(rng, 13, PIN.vocab)
    _, _, logits = oracle.prefill(PIN, W, prompt, cache_dtype=torch.float64)
    ref = hf_logits(model, prompt)
    assert (logits - ref).abs().max().item() < 1e-5


def test_mha_special_case():
    W = pin_weights(PIN_MHA, 12)
    model = hf_model(PIN_MHA, W)
    rng = np.random.default_rng(7)
    prompt = wl.random_tokens(rng, 6, PIN_MHA.vocab)
    parents = wl.level_tree([1, 3, 2, 2], rng)
    tokens = wl.random_tokens(rng, len(parents), PIN_MHA.vocab)
    r = run_verify(PIN_MHA, W, prompt, (tokens, parents))
    for i in range(len(parents)):
        ref = hf_logits(model, prompt + branch_tokens(tokens, parents, i))[-1]
        assert (r["logits"][i] - ref).abs().max().item() < 1e-5


def test_single_node_tree_is_one_decode_step(pin_setup):
    W, model = pin_setup
    rng = np.random.default_rng(8)
    prompt = wl.random_tokens(rng, 10, PIN.vocab)
    root = 5
    r = run_verify(PIN, W, prompt, ([root], [-1]))
    ref = hf_logits(model, prompt + [root])[-1]
    assert r["accepted_len"] == [0]
    assert r["next_token"] == [int(torch.argmax(ref))]
    assert r["path"] == [[0]]


def test_star_tree_is_independent_continuations(pin_setup):
    W, model = pin_setup
    rng = np.random.default_rng(9)
    prompt = wl.random_tokens(rng, 8, PIN.vocab)
    tokens = wl.random_tokens(rng, 7, PIN.vocab)
    parents = [-1] + [0] * 6
    r = run_verify(PIN, W, prompt, (tokens, parents))
    for c in range(1, 7):
        ref = hf_logits(model, prompt + [tokens[0], tokens[c]])[-1]
        assert (r["logits"][c] - ref).abs().max().item() < 1e-5


def test_greedy_draft_is_fully_accepted(pin_setup):
    W, model = pin_setup
    rng = np.random.default_rng(10)
    prompt = wl.random_tokens(rng, 8, PIN.vocab)
    greedy = hf_greedy(model, prompt, 7)
    # chain of the greedy tokens: everything accepted
    r = run_verify(PIN, W, prompt, (greedy[:6], wl.chain_tree(6)))
    assert r["accepted_len"] == [5] and r["next_token"] == [greedy[6]]
    assert r["path"] == [list(range(6))]
    # a tree whose deepest branch carries the greedy tokens
    parents = wl.recursive_tree(rng, 16, 5, 3)
    tokens = wl.random_tokens(rng, 16, PIN.vocab)
    branch = wl.deepest_branch(parents, rng)
    for lvl, node in enumerate(branch):
        tokens[node] = greedy[lvl]
    for i in range(1, 16):          # keep every other node off the greedy path
        if i not in branch and tokens[i] == greedy[wl.tree_depths(parents)[i]]:
            tokens[i] = (tokens[i] + 1) % PIN.vocab
    r = run_verify(PIN, W, prompt, (tokens, parents))
    assert r["accepted_len"] == [len(branch) - 1]
    assert r["path"] == [branch]
    assert r["next_token"] == [greedy[len(branch)]]
    # an all-wrong draft: nothing accepted, the bonus token is the root's greedy successor
    wrong = [greedy[0]] + [(greedy[1] + 1) % PIN.vocab] * 5
    r = run_verify(PIN, W, prompt, (wrong, [-1] + [0] * 5))
    assert r["accepted_len"] == [0] and r["next_token"] == [greedy[1]]


def test_chain_drafts_reproduce_greedy_decoding(pin_setup):
    """Several verify + commit rounds with perturbed greedy chain drafts give
    exactly the plain greedy token stream (lossless, Section 2.2)."""
    W, model = pin_setup
    rng = np.random.default_rng(11)
    prompt = wl.random_tokens(rng, 7, PIN.vocab)
    want = hf_greedy(model, prompt, 30)
    pk, pv, logits = oracle.prefill(PIN, W, prompt, cache_dtype=torch.float64)
    stream = [int(torch.argmax(logits[-1]))]
    ks, vs, lens = [pk], [pv], [len(prompt)]
    steps = 0
    while len(stream) < 26:
        n0 = len(stream)
        draft = [stream[-1]] + [want[n0 + j] if n0 + j < len(want) and rng.random() > 0.3
                                else int(rng.integers(PIN.vocab)) for j in range(3)]
        r = oracle.verify(PIN, W, ks, vs, lens, [(draft, wl.chain_tree(4))])
        acc = r["accepted_len"][0]
        assert r["path"][0] == list(range(acc + 1))      # chains never need moves
        stream += draft[1:acc + 1] + [r["next_token"][0]]
        ks, vs, lens = oracle.commit(ks, vs, lens, r, cache_dtype=torch.float64)
        assert lens[0] == len(prompt) + len(stream) - 1
        steps += 1
    assert stream[:26] == want[:26]
    assert steps < 26     # some drafts were accepted


def relabel(parents, rng):
    """A uniformly drawn topological order; returns (new parents, old id of each new id)."""
    T = len(parents)
    kids = [[] for _ in range(T)]
    for i in range(1, T):
        kids[parents[i]].append(i)
    order, frontier = [0], list(kids[0])
    while frontier:
        node = frontier.pop(int(rng.integers(len(frontier))))
        order.append(node)
        frontier += kids[node]
    new_of = {old: new for new, old in enumerate(order)}
    return [-1] + [new_of[parents[old]] for old in order[1:]], order


def test_relabelled_tree_permutes_results(pin_setup):
    W, _ = pin_setup
    rng = np.random.default_rng(12)
    prompt = wl.random_tokens(rng, 9, PIN.vocab)
    parents = wl.recursive_tree(rng, 14, 5, 3)
    tokens = wl.random_tokens(rng, 14, PIN.vocab)
    r = run_verify(PIN, W, prompt, (tokens, parents))
    parents2, old = relabel(parents, rng)
    assert parents2 != parents
    tokens2 = [tokens[o] for o in old]
    r2 = run_verify(PIN, W, prompt, (tokens2, parents2))
    for i in range(14):
        assert (r2["logits"][i] - r["logits"][old[i]]).abs().max().item() < 1e-12
    assert r["accepted_len"] == r2["accepted_len"]
    seq1 = [tokens[n] for n in r["path"][0]] + [r["next_token"][0]]
    seq2 = [tokens2[n] for n in r2["path"][0]] + [r2["next_token"][0]]
    assert seq1 == seq2


def test_verify_leaves_prefix_untouched(pin_setup):
    W, _ = pin_setup
    rng = np.random.default_rng(13)
    prompt = wl.random_tokens(rng, 9, PIN.vocab)
    pk, pv, _ = oracle.prefill(PIN, W, prompt, cache_dtype=torch.float64)
    pk0, pv0 = pk.clone(), pv.clone()
    parents = wl.recursive_tree(rng, 10, 4, 3)
    tokens = wl.random_tokens(rng, 10, PIN.vocab)
    r = oracle.verify(PIN, W, [pk], [pv], [9], [(tokens, parents)])
    assert torch.equal(pk, pk0) and torch.equal(pv, pv0)
    ks, vs, lens = oracle.commit([pk], [pv], [9], r, cache_dtype=torch.float64)
    assert torch.equal(ks[0][:, :, :9], pk0) and torch.equal(vs[0][:, :, :9], pv0)
    path = torch.tensor(r["path"][0])
    assert torch.equal(ks[0][:, :, 9:], r["tree_k"][0][:, :, path])
    assert lens == [9 + r["accepted_len"][0] + 1]


# ---------------------------------------------------------------------------
# the bf16-operand mode
# ---------------------------------------------------------------------------

def bf16_weights(W):
    """The same weights rounded to bf16 values (as the GPU holds them)."""
    r = lambda t: t.to(torch.bfloat16).to(torch.float64)   # noqa: E731
    return {"tok_embed": r(W["tok_embed"]), "final_norm": r(W["final_norm"]),
            "lm_head": r(W["lm_head"]),
            "layers": [{k: r(v) for k, v in lw.items()} for lw in W["layers"]]}


@pytest.fixture(scope="module")
def pin_setup_f64():
    W = bf16_weights(pin_weights(PIN, 21))
    return W, hf_model_f64(PIN, W)


def bf16_case(seed):
    rng = np.random.default_rng(300 + seed)
    prompt = wl.random_tokens(rng, 9, PIN.vocab)
    parents = wl.recursive_tree(rng, 18, 6, 3)
    tokens = wl.random_tokens(rng, len(parents), PIN.vocab)
    return prompt, tokens, parents


def test_exact_mode_matches_float64_decoder(pin_setup_f64):
    """With RMSNorm, rotary tables and softmax in float64 the decoder and the
    exact oracle agree to rounding order."""
    W, model = pin_setup_f64
    prompt, tokens, parents = bf16_case(0)
    r = run_verify(PIN, W, prompt, (tokens, parents))
    with bf16_storage(model, skip=STORAGE_POINTS):
        for i in range(len(parents)):
            ref = hf_logits(model, prompt + branch_tokens(tokens, parents, i))[-1]
            assert (r["logits"][i] - ref).abs().max().item() < 1e-12 * max(1.0, ref.abs().max().item())


def test_operand_mode_none_is_the_exact_path(pin_setup_f64):
    W, _ = pin_setup_f64
    prompt, tokens, parents = bf16_case(1)
    pk, pv, _ = oracle.prefill(PIN, W, prompt, cache_dtype=torch.float64)
    a = oracle.verify(PIN, W, [pk], [pv], [len(prompt)], [(tokens, parents)])
    for od in (None, torch.float64):
        b = oracle.verify(PIN, W, [pk], [pv], [len(prompt)], [(tokens, parents)], operand_dtype=od)
        assert torch.equal(a["logits"], b["logits"])
        assert torch.equal(a["tree_k"][0], b["tree_k"][0]) and torch.equal(a["tree_v"][0], b["tree_v"][0])


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_bf16_operand_mode_matches_rounded_decoder(pin_setup_f64, seed):
    """Every node's bf16-mode logits equal its branch decoded on its own by
    the decoder with the bf16 storage points rounded; leaving out any single
    rounding point (in the decoder) moves some logit by more than 1e-3, so an
    oracle that missed one would fail here."""
    W, model = pin_setup_f64
    prompt, tokens, parents = bf16_case(seed)
    bf = torch.bfloat16
    pk, pv, _ = oracle.prefill(PIN, W, prompt, cache_dtype=bf, operand_dtype=bf)
    r = oracle.verify(PIN, W, [pk], [pv], [len(prompt)], [(tokens, parents)], operand_dtype=bf)
    branches = [prompt + branch_tokens(tokens, parents, i) for i in range(len(parents))]
    with bf16_storage(model):
        ref = torch.stack([hf_logits(model, br)[-1] for br in branches])
    scale = ref.abs().max().item()
    assert (r["logits"] - ref).abs().max().item() < 1e-12 * scale
    # the K/V the bf16 mode stores are bf16 values
    assert torch.equal(r["tree_k"][0], r["tree_k"][0].to(bf).to(torch.float64))
    assert torch.equal(r["tree_v"][0], r["tree_v"][0].to(bf).to(torch.float64))
    for point in STORAGE_POINTS:
        with bf16_storage(model, skip=(point,)):
            alt = torch.stack([hf_logits(model, br)[-1] for br in branches])
        assert (r["logits"] - alt).abs().max().item() > 1e-3, point
