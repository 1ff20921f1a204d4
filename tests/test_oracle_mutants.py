"""The oracle's pins must catch plausible mistakes.  Each case plants one
mistake in a copy of the oracle's C source (on the CPU), builds it and runs
the pin suite against that build in a subprocess: the suite has to fail."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
LAYER_SRC, PLACE_SRC = "moe_oracle.c", "place_oracle.c"
PINS = {LAYER_SRC: os.path.join(ROOT, "tests", "test_oracle_pins.py"),
        PLACE_SRC: os.path.join(ROOT, "tests", "test_place_pins.py")}

# (name, text to replace, replacement, which occurrence (0-based))
MUTANTS = [
    ("order_reversed", "return a > b;", "return a < b;", 0),
    ("tie_to_higher_index", "return ia < ib;", "return ia > ib;", 1),
    ("nan_first", "return b_nan;", "return a_nan;", 0),
    ("gates_not_normalised", "exp((double)row[idx[j]] - m) / sum", "exp((double)row[idx[j]] - m)", 0),
    ("gate_sign", "sum += exp((double)row[idx[j]] - m);", "sum += exp(m - (double)row[idx[j]]);", 0),
    ("counts_transposed", "counts[(size_t)src[t] * E + e] += 1;", "counts[(size_t)e * S + src[t]] += 1;", 0),
    ("load_counts_sources", "expert_load[e] += 1;", "expert_load[src[t]] += 1;", 0),
    ("offsets_inclusive", "offsets[s + 1] = offsets[s] + (int32_t)fill[s];",
     "offsets[s + 1] = offsets[s] + (int32_t)fill[s] + (s == 0);", 0),
    ("unstable_within_slot", "int32_t r = offsets[s] + (int32_t)fill[s];",
     "int32_t r = offsets[s + 1] - 1 - (int32_t)fill[s];", 0),
    ("silu_sign", "return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));", 0),
    ("silu_is_relu", "return z / (1.0 + exp(-z));", "return z > 0 ? z : 0.0;", 0),
    ("gate_up_swapped", "h[i] = silu(g) * u;", "h[i] = silu(u) * g;", 0),
    ("down_transposed", "acc += bf16_value(row[c]) * v[c];",
     "acc += bf16_value(w[(size_t)c * n_out + (o % n_out)]) * v[c];", 0),
    ("dropped_last_term", "for (int c = 0; c < n_in; ++c)", "for (int c = 0; c + 1 < n_in; ++c)", 0),
    ("gate_weight_dropped", "o[c] += w[j] * y[c];", "o[c] += y[c];", 0),
    ("remote_experts_kept", "if (s < 0)\n                continue;\n            rc = oracle_swiglu_ffn",
     "if (s < 0)\n                s = idx[j] % E_local;\n            rc = oracle_swiglu_ffn", 0),
    ("shared_dropped", "for (int q = 0; q < n_sh; ++q) {", "for (int q = 0; q < 0; ++q) {", 0),
    ("combine_weight_dropped", "o[c] += w * bf16_value(", "o[c] += bf16_value(", 0),
    ("group_score_max_only", "gscore[q] = second < 0 ? c[first] : c[first] + c[second];", "gscore[q] = c[first];", 0),
    ("groups_worst_kept", "if (best < 0 || comes_before(gscore[q], q, gscore[best], best))",
     "if (best < 0 || comes_before(gscore[best], best, gscore[q], q))", 0),
    ("group_membership_strided", "allowed[e] = gtaken[e / gsz];", "allowed[e] = gtaken[e % n_group];", 0),
    ("sigmoid_sign", "exp(-(double)row[e])", "exp((double)row[e])", 0),
    ("bias_ignored", "c[e] = bias ? s + bias[e] : s;", "c[e] = s;", 0),
    ("bias_in_gates", "w[j] = sg[idx[j]] / sum;", "w[j] = (double)c[idx[j]] / sum;", 0),
    ("softmax_full_over_selected", "for (int e = 0; e < E; ++e)\n                sum += exp((double)row[e] - m);",
     "for (int e = 0; e < k; ++e)\n                sum += exp((double)row[idx[e]] - m);", 0),
    ("scale_dropped", "w[j] *= scale;", "w[j] *= 1.0;", 0),
]
LAYER_MUTANTS = [(LAYER_SRC,) + m for m in MUTANTS]

PLACE_MUTANTS = [(PLACE_SRC,) + m for m in [
    ("coldest_first", "return Ba > Bb;", "return Ba < Bb;", 0),
    ("volume_ignored", "return Va > Vb;", "return a < b;", 0),
    ("load_term_sign", "double c_load = v * v - u * u;", "double c_load = u * u - v * v;", 0),
    ("load_term_without_expert", "double v = (double)(load[g] + Bl[e]) - mean;",
     "double v = (double)load[g] - mean;", 0),
    ("load_term_absolute", "double c_load = v * v - u * u;", "double c_load = v * v;", 0),
    ("mean_over_experts", "double mean = (double)total / G;", "double mean = (double)total / E;", 0),
    ("old_rank_not_charged", "c_mig = c_mig + mig_cost(M, m_uniform, l, E, G, e, home);",
     "c_mig = c_mig + 0.0;", 0),
    ("comm_d_transposed", "(double)Al[(size_t)s * E + e] * D[(size_t)s * G + g];",
     "(double)Al[(size_t)s * E + e] * D[(size_t)(g % S) * G + (s % G)];", 0),
    ("comm_a_transposed", "c_comm = c_comm + (double)Al[(size_t)s * E + e]",
     "c_comm = c_comm + (double)Al[(size_t)(e % S) * E + (s % E)]", 0),
    ("tie_prefers_moving", "take = g == home;", "take = g != home;", 0),
    ("tie_prefers_fuller", "take = n[g] < n[best];", "take = n[g] > n[best];", 0),
    ("tie_to_higher_rank", "take = g < best;", "take = g > best;", 0),
    ("capacity_off_by_one", "if (n[g] >= cap[g])", "if (n[g] > cap[g])", 0),
    ("nan_wins", "score = INFINITY;", "score = -INFINITY;", 0),
    ("beta_dropped", "score = score + beta * c_load;", "score = score + c_load;", 0),
    ("objective_mean_wrong", "mean /= G;", "mean /= (G + 1);", 0),
    ("objective_mig_signed", "* fabs(xi - x0i);", "* (xi - x0i);", 0),
    ("window_home_inverted", "if (xl[e] != home[s] || home[s] < 0", "if (xl[e] == home[s] || home[s] < 0", 0),
    ("window_total_only_remote", "tot += a;", "tot += a * (xl[e] != home[s]);", 0),
    ("window_load_one_source", "                        b += Al[(size_t)s * E + e];",
     "                        b += Al[e];", 0),
    ("window_b_ignored", "b = B[(size_t)l * E + e];", "b = Al[e];", 0),
    ("window_pressure_raw", "pressure[d] / mean;", "pressure[d];", 0),
    ("window_engine_ignored", "if ((engine ? engine[g] : g) == d)", "if (g == d)", 0),
    ("objective_comm_ignores_x", "D[(size_t)s * G + g] *\n                              (xl[e] == g ? 1.0 : 0.0);",
     "D[(size_t)s * G + g] *\n                              (xl[e] == g ? 1.0 : 1.0);", 0),
]]


def _mutate(src: str, old: str, new: str, nth: int) -> str:
    pos = -1
    for _ in range(nth + 1):
        pos = src.find(old, pos + 1)
        assert pos >= 0, f"pattern not found: {old!r}"
    return src[:pos] + new + src[pos + len(old):]


ALL = LAYER_MUTANTS + PLACE_MUTANTS


@pytest.mark.parametrize("src_name,name,old,new,nth", ALL, ids=[m[1] for m in ALL])
def test_pins_catch_mutant(tmp_path, src_name, name, old, new, nth):
    sources = []
    for fname in (LAYER_SRC, PLACE_SRC):
        with open(os.path.join(ORACLE, fname)) as f:
            src = f.read()
        if fname == src_name:
            mutated = _mutate(src, old, new, nth)
            assert mutated != src
            src = mutated
        c = tmp_path / fname
        c.write_text(src)
        sources.append(str(c))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fPIC", "-shared", *sources,
                           "-o", str(so), "-lm"])
    env = dict(os.environ, MOE_ORACLE_LIB=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", PINS[src_name]],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 1, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
