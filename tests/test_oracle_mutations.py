"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a temporary copy of the oracle (on the CPU)
and runs the pin suite against that copy; the suite must fail.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = {
    "rotary sign": ("return torch.cat([a * c - b * s, b * c + a * s], dim=-1)",
                    "return torch.cat([a * c + b * s, b * c - a * s], dim=-1)"),
    "rotary frequency": ("theta ** (-2.0 * j / head_dim)", "theta ** (-1.0 * j / head_dim)"),
    "kv head of a query head": ("kv = h // group", "kv = h % n_kv_heads"),
    "norm gain dropped": ("keepdim=True) + eps) * gain", "keepdim=True) + eps)"),
    "position = S + node index": ('"pos": S + depth,', '"pos": S + torch.arange(len(tokens)),'),
    "siblings visible": ("anc[i] = anc[p]\n", "anc[i] = anc[p] | anc[i - 1]\n"),
    "score scale dropped": ("@ k_all[kv].T) / math.sqrt(d)", "@ k_all[kv].T)"),
    "gate and up swapped": ("silu(gate) * up)", "silu(up) * gate)"),
    "ffn residual dropped": ("x = x + rnd(torch.nn.functional.silu(gate) * up) @",
                             "x = rnd(torch.nn.functional.silu(gate) * up) @"),
    "softmax not normalised": ("/ e.sum(dim=-1, keepdim=True)", ""),
    "mask not applied": ('s = s.masked_fill(~visible, float("-inf"))', "s = s"),
    "deepest-node tie toward higher index": ("depth[i] > depth[best]", "depth[i] >= depth[best]"),
    "acceptance ignores the parent": ("accepted[i] = accepted[p] and", "accepted[i] ="),
    # rounding points of the bf16-operand mode
    "bf16: attention norm output not rounded": (
        'h = rnd(rms_norm(x, _f64(lw["attn_norm"]), cfg.rms_eps))',
        'h = rms_norm(x, _f64(lw["attn_norm"]), cfg.rms_eps)'),
    "bf16: v not rounded": ('v = rnd((h @ _f64(lw["wv"]).T).view(N, nkv, d))',
                            'v = (h @ _f64(lw["wv"]).T).view(N, nkv, d)'),
    "bf16: q not rounded": ("q = rnd(rope(q, cos, sin))", "q = rope(q, cos, sin)"),
    "bf16: k rounded before the rotation": (
        ['k = (h @ _f64(lw["wk"]).T).view(N, nkv, d)', "k = rnd(rope(k, cos, sin))"],
        ['k = rnd((h @ _f64(lw["wk"]).T).view(N, nkv, d))', "k = rope(k, cos, sin)"]),
    "bf16: softmax numerators not rounded": ("(rnd(e) @ v_all[kv])", "(e @ v_all[kv])"),
    "bf16: normalised weights rounded": (
        "(rnd(e) @ v_all[kv]) / e.sum(dim=-1, keepdim=True)",
        "rnd(e / e.sum(dim=-1, keepdim=True)) @ v_all[kv]"),
    "bf16: attention output not rounded": ("x = x + rnd(o.reshape(N, nq * d)) @",
                                           "x = x + o.reshape(N, nq * d) @"),
    "bf16: ffn norm output not rounded": (
        'h2 = rnd(rms_norm(x, _f64(lw["ffn_norm"]), cfg.rms_eps))',
        'h2 = rms_norm(x, _f64(lw["ffn_norm"]), cfg.rms_eps)'),
    "bf16: activation not rounded": ("x = x + rnd(torch.nn.functional.silu(gate) * up) @",
                                     "x = x + (torch.nn.functional.silu(gate) * up) @"),
    "bf16: final norm output not rounded": (
        'hf = rnd(rms_norm(x, _f64(W["final_norm"]), cfg.rms_eps))',
        'hf = rms_norm(x, _f64(W["final_norm"]), cfg.rms_eps)'),
}


@pytest.mark.slow
@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(tmp_path, name):
    before, after = MUTATIONS[name]
    for d in ("oracle", "workload", "tests"):
        shutil.copytree(os.path.join(ROOT, d), tmp_path / d,
                        ignore=shutil.ignore_patterns("__pycache__", "golden"))
    src = (tmp_path / "oracle" / "verify.py").read_text()
    for b, a in zip(*((before, after) if isinstance(before, list) else ([before], [after]))):
        assert src.count(b) == 1, (name, b)
        src = src.replace(b, a)
    (tmp_path / "oracle" / "verify.py").write_text(src)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "tests/test_oracle_pins.py"], cwd=tmp_path, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode != 0, f"pins did not catch: {name}\n{r.stdout[-2000:]}"
