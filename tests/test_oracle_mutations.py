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
    "norm gain dropped": ("+ eps) * gain", "+ eps)"),
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
}


@pytest.mark.slow
@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(tmp_path, name):
    before, after = MUTATIONS[name]
    for d in ("oracle", "workload", "tests"):
        shutil.copytree(os.path.join(ROOT, d), tmp_path / d,
                        ignore=shutil.ignore_patterns("__pycache__", "golden"))
    src = (tmp_path / "oracle" / "verify.py").read_text()
    assert before in src, name
    (tmp_path / "oracle" / "verify.py").write_text(src.replace(before, after))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "tests/test_oracle_pins.py"], cwd=tmp_path, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode != 0, f"pins did not catch: {name}\n{r.stdout[-2000:]}"
