"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle source (dropped term,
wrong sign or index, transposed operand, wrong tie rule, ...), builds it with
gcc into a temporary directory, and runs the oracle pin tests against that
build.  The suite must fail for every mutant.  Nothing here touches the GPU.
"""
import os
import subprocess
import sys

import pytest

import oracle.oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_TESTS = ["tests/test_oracle_route.py", "tests/test_oracle_dispatch_prune.py",
             "tests/test_oracle_forward.py", "tests/test_oracle_shared.py",
             "tests/test_oracle_mass.py"]

# (name, original text, mutated text); every occurrence is replaced.
MUTANTS = [
    ("gate_up_swapped", "const uint16_t* up = gate + I * H;",
     "const uint16_t* up = gate; gate = gate + I * H;"),
    ("down_transposed", "down[o * I + i]", "down[i * H + o]"),
    ("silu_sign", "expf(-g)", "expf(g)"),
    ("silu_dropped", "return (g / (1.0f + expf(-g))) * u;", "return g * u;"),
    ("no_renormalisation", "w[j] = w[j] / denom;", "w[j] = w[j];"),
    ("softmax_sign", "w[j] = expf(z[ids[j]] - zmax);", "w[j] = expf(zmax - z[ids[j]]);"),
    ("topk_tie_to_larger_id", "if (best < 0 || z[e] > z[best]) best = e;",
     "if (best < 0 || z[e] >= z[best]) best = e;"),
    ("topk_picks_smallest", "if (best < 0 || z[e] > z[best]) best = e;",
     "if (best < 0 || z[e] < z[best]) best = e;"),
    ("router_transposed", "acc += widen_bf16(xt[hh]) * we[hh];",
     "acc += widen_bf16(xt[hh]) * wr[(size_t)hh * n_experts + e];"),
    ("bias_dropped", "if (bias) acc += bias[e];", ""),
    ("mask_ignored", "taken[e] = (keep_mask && !keep_mask[e]) ? 1 : 0;", "taken[e] = 0;"),
    ("gap_wrong_rank", "z[ids[top_k - 1]] - z[next]", "z[ids[0]] - z[next]"),
    ("combine_wrong_gate", "const float wj = topk_w[(size_t)t * top_k + j];",
     "const float wj = topk_w[(size_t)t * top_k];"),
    ("combine_overwrites", "ot[o] += wj * y;", "ot[o] = wj * y;"),
    ("dropped_last_hidden_term", "for (size_t h = 0; h < H; ++h) {\n          const float xv",
     "for (size_t h = 0; h + 1 < H; ++h) {\n          const float xv"),
    ("dropped_last_inter_term", "for (size_t i = 0; i < I; ++i) y += widen_bf16",
     "for (size_t i = 0; i + 1 < I; ++i) y += widen_bf16"),
    ("dispatch_offsets_inclusive", "    offsets[e] = pos;\n", "    offsets[e] = pos + 1;\n"),
    ("dispatch_active_all", "if (c > 0) active[na++] = e;", "active[na++] = e;"),
    ("prune_ties_to_larger_id", "importance[order[j]] < importance[cur]",
     "importance[order[j]] <= importance[cur]"),
    ("prune_keeps_lowest", "importance[order[j]] < importance[cur]",
     "importance[order[j]] > importance[cur]"),
    ("compact_wrong_rows", "memcpy(w13_c + ci * 2 * in * h, w13 + e * 2 * in * h",
     "memcpy(w13_c + ci * 2 * in * h, w13 + ci * 2 * in * h"),
    ("bf16_widen_wrong_shift", "((uint32_t)bits) << 16", "((uint32_t)bits) << 15"),
    ("shared_gate_sign", "const float s = 1.0f / (1.0f + expf(-z));",
     "const float s = 1.0f / (1.0f + expf(z));"),
    ("shared_overwrites", "ot[o] += s * y;", "ot[o] = s * y;"),
    ("shared_up_is_gate", "const uint16_t* up = w13 + I * H;", "const uint16_t* up = w13;"),
    ("mass_no_shift", "denom += expf(zt[e] - zmax);", "denom += expf(zt[e]);"),
    ("mass_ignores_mask", "if ((!keep_mask || keep_mask[e]) && zt[e] > zmax) zmax = zt[e];",
     "if (zt[e] > zmax) zmax = zt[e];"),
    ("mass_topk_unweighted", "mass_topk[ids[t * k + j]] += w[t * k + j];",
     "mass_topk[ids[t * k + j]] += 1.0f;"),
]


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(name, orig, mut, tmp_path):
    with open(O._SRC) as f:
        src = f.read()
    assert orig in src, f"mutation anchor for {name} not found in the oracle source"
    mutated = src.replace(orig, mut)
    d = tmp_path / "oracle_src"
    d.mkdir()
    (d / "slimwise_oracle.c").write_text(mutated)
    with open(os.path.join(os.path.dirname(O._SRC), "swo.h")) as f:
        (d / "swo.h").write_text(f.read())
    so = tmp_path / "libswo_mut.so"
    subprocess.check_call(["gcc", *O.CFLAGS, "-o", str(so), str(d / "slimwise_oracle.c"), "-lm"])
    env = dict(os.environ, SWO_LIB=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *PIN_TESTS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the oracle pins:\n{r.stdout[-2000:]}"
