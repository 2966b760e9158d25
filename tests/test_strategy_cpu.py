"""The library's cost predictor and draft-token-num selection (host code
behind the C ABI) against the oracle: same n, same selection order, same
objectives; validation of malformed calls."""

import numpy as np
import pytest

import paper_2512_04752_amd as sv
from oracle import strategy as S
from tests.test_oracle_strategy import monotone_weights, random_tree


def flat(trees):
    offs = np.zeros(len(trees) + 1, dtype=np.int32)
    offs[1:] = np.cumsum([len(p) for p, _ in trees])
    return offs, [x for p, _ in trees for x in p], [x for _, w in trees for x in w]


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("bucket", [0.0, 0.05])
def test_selection_matches_oracle(seed, bucket):
    rng = np.random.default_rng(500 + seed)
    trees = []
    for _ in range(int(rng.integers(1, 17))):
        p = random_tree(rng, int(rng.integers(1, 90)), max_children=4)
        w = np.float32(monotone_weights(rng, p)).astype(np.float64).tolist()   # float32 like the ABI
        trees.append((p, w))
    lens = [int(x) for x in rng.integers(0, 30000, len(trees))]
    coeffs = {"c0": float(rng.uniform(2, 8)), "c_seq": float(rng.uniform(5e-6, 5e-5)),
              "c_draft": float(rng.uniform(0.005, 0.05)), "c_tree": float(rng.uniform(0, 1e-7)),
              "bucket_ratio": bucket}
    n_max, patience = int(rng.integers(4, 65)), int(rng.integers(1, 4))
    model = sv.CostModel.from_dict(coeffs)
    offs, pars, ws = flat(trees)
    n, sel, obj = sv.spec_select_draft_count(model, lens, offs, pars, ws, n_max, patience)
    n_or, seen = S.select(coeffs, lens, trees, n_max, patience)
    assert n == n_or
    assert np.allclose(obj[:len(seen)], seen, rtol=1e-9)
    assert (obj[len(seen):] == 0).all()
    for b, (p, w) in enumerate(trees):
        order = S.selection_order(p, w)[:n_max]
        assert sel[b, :len(order)].tolist() == order
        assert (sel[b, len(order):] == -1).all()


def test_predictor_matches_oracle_and_caches():
    coeffs = {"c0": 4.1, "c_seq": 2.3e-5, "c_draft": 0.0171, "c_tree": 9e-8, "bucket_ratio": 0.1}
    m = sv.CostModel.from_dict(coeffs)
    rng = np.random.default_rng(2)
    for _ in range(200):
        ns, nd = int(rng.integers(0, 800000)), int(rng.integers(0, 20000))
        tk = ns * int(rng.integers(1, 65))
        assert m.predict(ns, nd, tk) == pytest.approx(S.cost(coeffs, ns, nd, tk), rel=1e-12)
    hits, misses = m.stats()
    assert hits + misses == 200 and misses < 200
    exact = sv.CostModel.from_dict(coeffs, bucket_ratio=0.0)
    assert exact.predict(1000, 8, 8000) == pytest.approx(4.1 + 0.023 + 0.1368 + 0.00072)


@pytest.mark.parametrize("case", ["root_parent", "order", "increasing", "negative", "n_max",
                                  "empty"])
def test_selection_validation(case):
    m = sv.CostModel(4.0, 1e-5, 0.01, 0.0)
    offs, pars, w, n_max = [0, 3], [-1, 0, 0], [1.0, 0.5, 0.4], 8
    if case == "root_parent":
        pars = [0, 0, 0]
    elif case == "order":
        pars = [-1, 2, 0]
    elif case == "increasing":
        w = [1.0, 0.5, 1.2]
    elif case == "negative":
        w = [1.0, -0.1, 0.2]
    elif case == "n_max":
        n_max = sv.SPEC_MAX_TREE + 1
    elif case == "empty":
        offs, pars, w = [0, 0], [], []
    with pytest.raises(sv.SpecError):
        sv.spec_select_draft_count(m, [100], offs, pars, w, n_max)


def test_bucket_ratio_validated():
    with pytest.raises(sv.SpecError):
        sv.CostModel(1, 0, 0, 0, bucket_ratio=2.0)


def test_product_fit_matches_oracle_fit_on_exact_data():
    from paper_2512_04752_amd import cost_fit
    rng = np.random.default_rng(8)
    truth = {"c0": 4.2, "c_seq": 1.8e-5, "c_draft": 0.017, "c_tree": 2e-8}
    rows = []
    for B in (1, 4, 16, 64, 256):
        for n in (1, 4, 8, 16, 32, 64):
            ns = int(B * rng.integers(500, 3000))
            ms = truth["c0"] + truth["c_seq"] * ns + truth["c_draft"] * B * n + truth["c_tree"] * n * ns
            rows.append({"batch": B, "budget": n, "tokens": B * n, "kv_tokens": ns + B * n,
                         "ms_per_step": ms, "accepted_tokens_per_s": B * n * 10.0})
    beta, loo = cost_fit.fit(rows)
    ref = S.fit([(*cost_fit.features(r), r["ms_per_step"]) for r in rows])
    assert np.allclose(beta, ref, rtol=1e-6)
    assert np.allclose(beta, [truth[k] for k in ("c0", "c_seq", "c_draft", "c_tree")], rtol=1e-6)
    assert max(abs(e) for e in loo) < 1e-6


def test_committed_cost_model_reproduces_from_committed_sweep():
    import json
    import os
    from paper_2512_04752_amd import cost_fit
    d = os.path.join(os.path.dirname(sv.__file__), "data")
    rows = [json.loads(l) for l in open(os.path.join(d, "verify_cost_sweep__llama8b_mi355x.jsonl"))]
    model = json.load(open(os.path.join(d, "verify_cost_model__llama8b_mi355x.json")))
    beta, _ = cost_fit.fit(rows)
    assert np.allclose(beta, [model[k] for k in ("c0", "c_seq", "c_draft", "c_tree")], rtol=1e-9,
                       atol=1e-15)
    assert all(model[k] >= 0 for k in ("c0", "c_seq", "c_draft", "c_tree"))
