"""Mutation check of the pins: plant one plausible mistake at a time in a copy of
the oracle's C source (CPU only), build it, and require the pin battery to reject
it.  A mutant that passes every pin would mean that part of the oracle is not
pinned.  Mutations are chosen so that the broken build still stays in bounds."""
import os
import subprocess

import pytest

import oracle
from oracle_pins import ALL_PINS

SRC = os.path.join(os.path.dirname(oracle.__file__), "omnimem_oracle.c")

# (name, exact text in the source, replacement)
MUTANTS = [
    ("pool_divides_by_B", "kbar[((int64_t)h * nb + b) * d + j] = sum / count;",
     "kbar[((int64_t)h * nb + b) * d + j] = sum / B;"),
    ("tail_block_drops_last_token", "int end = begin + B < S ? begin + B : S;",
     "int end = begin + B < S ? begin + B : S - 1;"),
    ("proxy_query_sum_not_mean", "qbar[(((int64_t)h * R) + r) * d + j] = sum / (q1 - q0);",
     "qbar[(((int64_t)h * R) + r) * d + j] = sum;"),
    ("group_boundary_off_by_one", "int q0 = r * G_q, q1 = q0 + G_q < Lq ? q0 + G_q : Lq;",
     "int q0 = r * G_q, q1 = q0 + G_q < Lq ? q0 + G_q + 1 : Lq;"),
    ("awe_chunk_threshold_strict", "return (outside_chunks >= T_out && outside_blocks >= K) ? 1 : 0;",
     "return (outside_chunks > T_out && outside_blocks >= K) ? 1 : 0;"),
    ("awe_block_guard_strict", "return (outside_chunks >= T_out && outside_blocks >= K) ? 1 : 0;",
     "return (outside_chunks >= T_out && outside_blocks > K) ? 1 : 0;"),
    ("awe_block_guard_dropped", "return (outside_chunks >= T_out && outside_blocks >= K) ? 1 : 0;",
     "return (outside_chunks >= T_out) ? 1 : 0;"),
    ("window_off_by_one", "int in_window = c >= n - E;", "int in_window = c > n - E;"),
    ("window_uses_offset_not_chunk", "int c = (int)(b / Bpc);\n    int in_window", "int c = (int)(b % Bpc);\n    int in_window"),
    ("residency_ignored_in_selection", "int is_resident = resident == NULL ? 1 : (resident[b] != 0);",
     "int is_resident = 1;"),
    ("ranking_reversed", "if (a->s > b->s) return -1;\n  if (a->s < b->s) return 1;",
     "if (a->s > b->s) return 1;\n  if (a->s < b->s) return -1;"),
    ("tie_break_reversed", "return (a->b < b->b) ? -1 : (a->b > b->b);", "return (a->b > b->b) ? -1 : (a->b < b->b);"),
    ("output_not_sorted_by_id", "qsort(chosen, (size_t)take, sizeof(int32_t), id_cmp);", ";"),
    ("score_unscaled", "double sb = scale * dot;", "double sb = dot;"),
    ("logit_unscaled", "logit_buf[i] = scale * dot;", "logit_buf[i] = dot;"),
    ("lse_missing_max", "*lse = mx + log(denom);", "*lse = log(denom);"),
    ("values_read_from_keys", "out[j] += w * widen(V, kv_at", "out[j] += w * widen(K, kv_at"),
    ("kv_layout_transposed", "return (((int64_t)c * S + t) * H + h) * d + j;", "return (((int64_t)c * S + t) * d + j) * H + h;"),
    ("residency_ignored_in_attention", "if (resident != NULL && !resident[b]) return nk;", "if (0) return nk;"),
    ("sparse_uses_first_group", "int h = hs[i], q = qs[i], r = q / G_q;", "int h = hs[i], q = qs[i], r = 0;"),
    ("dense_drops_last_chunk", "for (int32_t b = c0 * Bpc; b < c1 * Bpc; ++b)", "for (int32_t b = c0 * Bpc; b < (c1 - 1) * Bpc; ++b)"),
    ("softmax_not_normalised", "for (int j = 0; j < d; ++j) out[j] /= denom;", ";"),
    ("bf16_widened_wrong", "uint32_t bits = ((uint32_t)((const uint16_t*)base)[i]) << 16;",
     "uint32_t bits = ((uint32_t)((const uint16_t*)base)[i]) << 15;"),
    ("prob_lse_missing_max", "double lse_q = mx + log(denom);", "double lse_q = log(denom);"),
    ("prob_sum_not_mean", "double sb = sbar[b] / (double)(row1 - row0);", "double sb = sbar[b];"),
    ("prob_averages_logits", "sbar[b] += exp(u[b] - lse_q);", "sbar[b] += u[b];"),
    ("prob_softmax_over_omega_only", "for (int64_t b = 0; b < nb; ++b) denom += exp(u[b] - mx);",
     "for (int64_t b = 0; b < nb; ++b) denom += omega[b] ? exp(u[b] - mx) : 0.0;"),
    ("prob_group_rows_off_by_one", "row1 = row0 + G_q < Lq ? row0 + G_q : Lq;",
     "row1 = row0 + G_q < Lq ? row0 + G_q + 1 : Lq;"),
    ("prob_omega_ignored", "if (omega[b] != 0) {", "if (1) {"),
    ("union_counts_duplicates", "if (!mine[b]) { mine[b] = 1; ++count; }", "{ mine[b] = 1; ++count; }"),
]


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(name, old, new, source, tmp_path):
    assert source.count(old) >= 1, f"mutation site for {name} not found in the oracle source"
    mutated = source.replace(old, new, 1)
    src = tmp_path / "mutant.c"
    src.write_text(mutated)
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-w", "-o", str(so), str(src), "-lm"])
    caught = []
    with oracle.using_library(str(so)):
        for pin in ALL_PINS:
            try:
                pin()
            except (AssertionError, ValueError, ZeroDivisionError, FloatingPointError):
                caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"


# Mistakes planted in the oracle's Python-level functions: the function's source is
# edited, compiled in the oracle module's namespace and swapped in for the pins' run.
PY_MUTANTS = [
    ("gate_sigmoid_of_twice_the_logit", "gated_combine",
     "z = np.exp(-np.abs(gl[..., c]))", "z = np.exp(-2.0 * np.abs(gl[..., c]))"),
    ("gate_branches_reversed", "gated_combine", "z = np.exp(-np.abs(gl[..., c]))",
     "z = np.exp(-np.abs(gl[..., 2 - c]))"),
    ("gate_sign_flipped", "gated_combine", "np.where(gl[..., c] >= 0, 1.0 / (1.0 + z), z / (1.0 + z))",
     "np.where(gl[..., c] >= 0, z / (1.0 + z), 1.0 / (1.0 + z))"),
    ("bf16_rounds_to_7_bits", "round_bf16", "np.round(m * 256.0) / 256.0", "np.round(m * 128.0) / 128.0"),
    ("cmp_cache_values_from_keys", "cmp_cache", "kc, vc = pool_keys(k, B), pool_keys(v, B)",
     "kc, vc = pool_keys(k, B), pool_keys(k, B)"),
    ("lru_evicts_most_recent", "lru_simulate", "victim = next(v for v in order if v not in want)",
     "victim = next(v for v in reversed(order) if v not in want)"),
    ("lru_hits_do_not_refresh", "lru_simulate", "                order.remove(c)\n                order.append(c)\n",
     ""),
    ("lru_evicts_with_free_slots", "lru_simulate", "if free:", "if free and not slot_of:"),
    ("lru_highest_free_slot", "lru_simulate", "s = free[0]", "s = free[-1]"),
]


@pytest.mark.parametrize("name,func,old,new", PY_MUTANTS, ids=[m[0] for m in PY_MUTANTS])
def test_pins_reject_python_mutant(name, func, old, new, monkeypatch):
    import inspect
    import textwrap

    src = textwrap.dedent(inspect.getsource(getattr(oracle, func)))
    assert src.count(old) >= 1, f"mutation site for {name} not found in oracle.{func}"
    ns = dict(vars(oracle))
    exec(compile(src.replace(old, new, 1), f"<mutant {name}>", "exec"), ns)
    monkeypatch.setattr(oracle, func, ns[func])
    caught = []
    for pin in ALL_PINS:
        try:
            pin()
        except (AssertionError, ValueError, ZeroDivisionError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
