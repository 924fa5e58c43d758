"""Planted mistakes in the oracle are caught by its pins.

Each case copies ``oracle/oracle.c`` to a temporary directory, plants one
plausible mistake (a dropped term, a wrong sign, index or stride, a
transposed operand, a narrower accumulator, a wrong row count), builds it,
and runs the pin battery against it: at least one pin must fail.  The real
oracle must pass the same battery.
"""
import os
import subprocess

import pytest

import oracle
import test_oracle_bruteforce as bf
import test_oracle_invariants as inv
import test_oracle_multi as multi
import test_oracle_pins as pins
import test_oracle_vs_sdpa as sdpa

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "dropped_scale": ("s[l] = scale * dot;", "s[l] = dot;"),
    "exp_sign": ("++l) e[l] = exp(s[l] - m);", "++l) e[l] = exp(m - s[l]);"),
    "no_normalisation": ("e[l] = e[l] / Z;   /* e now holds a */", "(void)Z;"),
    "head_map_modulo": ("return (int)(((int64_t)h * h_kv) / h_q);", "return h % h_kv;"),
    "k_transposed": ("dot += (double)q[j] * (double)Krow[j];",
                     "dot += (double)q[j] * (double)Kslab[(int64_t)j * n + l];"),
    "v_row_stride_dk": ("const float *Vrow = Vslab + l * (int64_t)d_v;",
                        "const float *Vrow = Vslab + l * (int64_t)d_k;"),
    "float_accumulator": ("double dot = 0.0;", "float dot = 0.0f;"),
    "one_row_short": ("if (len_b > n_max) return n_max;\n    return len_b;",
                      "if (len_b > n_max) return n_max;\n    return len_b > 0 ? len_b - 1 : 0;"),
    "one_row_long": ("if (len_b > n_max) return n_max;\n    return len_b;",
                     "if (len_b >= n_max) return n_max;\n    return len_b + 1;"),
    "append_no_increment": ("        len[b] = t + 1;\n    }\n    return 0;",
                            "        (void)0;\n    }\n    return 0;"),
    "append_wrong_row": ("memcpy(Ks + (int64_t)t * d_k, k_new + ((int64_t)b * h_kv + g) * d_k,",
                         "memcpy(Ks + (int64_t)(t > 0 ? t - 1 : 0) * d_k, k_new + ((int64_t)b * h_kv + g) * d_k,"),
    "max_not_subtracted_wrongly": ("if (s[l] > m) m = s[l];", "if (s[l] < m || m == -INFINITY) m = s[l];\n        m = 0.0;"),
    "multi_sees_next_row": ("const int64_t pos = rows_used(len[b], n_max) - T + r;",
                            "const int64_t pos = rows_used(len[b], n_max) - T + r + 1;"),
    "multi_rows_reversed": ("const int64_t pos = rows_used(len[b], n_max) - T + r;",
                            "const int64_t pos = rows_used(len[b], n_max) - 1 - r;"),
    "multi_query_stride": ("const float *qv = q + u * d_k;", "const float *qv = q + bh * d_k;"),
    "append_rows_reversed": ("const int64_t src = ((int64_t)b * h_kv + g) * T + r;",
                             "const int64_t src = ((int64_t)b * h_kv + g) * T + (T - 1 - r);"),
}


def _battery():
    """Fast pins from every pin module; returns the names that failed."""
    checks = [
        pins.test_worked_decode_example_matches_printed_values,
        pins.test_worked_decode_example_closed_form,
        pins.test_gamma_offsets_are_the_layout_both_sides_read,
        pins.test_append_example_writes_offsets_6_7_8_only,
        lambda: pins.test_gqa_head_map({"h_q": 4, "h_kv": 2, "kv_head_of": [0, 0, 1, 1]}),
        pins.test_rows_beyond_len_are_not_read,
        lambda: bf.test_oracle_matches_decimal_bruteforce(bf.CASES[2], 0),
        lambda: bf.test_oracle_matches_decimal_bruteforce(bf.CASES[3], 1),
        bf.test_bruteforce_catches_large_logits,
        lambda: inv.test_weights_sum_to_one(0),
        inv.test_single_row_returns_that_row_exactly,
        inv.test_append_then_decode_equals_decode_on_full_cache,
        lambda: sdpa.test_table3_multistep_kv_cache_vs_causal_sdpa({"T": 4, "d": 8}),
        lambda: multi.test_longer_cache_equals_masked_sdpa(4, [37, 9]),
        multi.test_equals_t_single_steps_bit_for_bit,
        multi.test_append_rows_offsets_and_capacity,
    ]
    failed = []
    for i, c in enumerate(checks):
        try:
            c()
        except (AssertionError, ValueError, TypeError):
            failed.append(i)
    return failed


def _build(tmp_path, src_text, name):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"lib{name}.so"
    c.write_text(src_text)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    "-o", str(so), str(c), "-lm"], check=True)
    return str(so)


def test_unmodified_oracle_passes_the_battery(tmp_path):
    src = open(SRC).read()
    with oracle.use_library(_build(tmp_path, src, "clean")):
        assert _battery() == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    src = open(SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    with oracle.use_library(_build(tmp_path, src.replace(old, new), name)):
        assert _battery(), f"no pin caught the planted mistake {name}"
