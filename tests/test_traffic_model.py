"""The byte-accounting functions the benchmark uses reproduce the paper's
traffic tables (Tables 2, 4, 6; MB = 1e6 bytes, 2 printed decimals)."""
import json
import os

import pytest

from paper_2607_19456_amd import traffic

with open(os.path.join(os.path.dirname(__file__), "golden", "traffic_tables.json")) as f:
    TABLES = json.load(f)


def _mb(x):
    return round(x / 1e6, 2)


@pytest.mark.parametrize("row", TABLES["table2"], ids=lambda r: f"n{r['n']}")
def test_table2(row):
    assert _mb(traffic.decode_bytes(row["n"], 64, 64)) == row["moa_MB"]
    assert _mb(traffic.score_matrix_bytes(row["n"])) == row["n2_MB"]


@pytest.mark.parametrize("row", TABLES["table4"], ids=lambda r: f"T{r['T']}")
def test_table4(row):
    app, dec, n2 = traffic.multistep_table(row["T"], 64, 64)
    assert (_mb(app), _mb(dec), _mb(n2)) == (row["app_MB"], row["dec_MB"], row["n2_MB"])


def test_table4_ratio_claim():
    c = TABLES["table4_ratio_claim"]
    app, dec, n2 = traffic.multistep_table(c["T"], 64, 64)
    assert round(n2 / (app + dec), 1) == c["ratio"]


@pytest.mark.parametrize("row", TABLES["table6"], ids=lambda r: f"hkv{r['h_kv']}")
def test_table6(row):
    kv, total = traffic.gqa_table(1024, 64, 64, 32, row["h_kv"])
    assert (_mb(kv), _mb(total)) == (row["kv_MB"], row["total_MB"])


def test_eq8_step_cost_sums_to_table4_order():
    # eq. (8) summed over steps is O(T^2 (d_k+d_v)) and matches Table 4's
    # decode column up to the query/output terms Proposition 1 adds per step.
    T, d = 64, 64
    eq8 = sum(traffic.step_bytes(t, d, d) for t in range(1, T + 1))
    app, dec, _ = traffic.multistep_table(T, d, d)
    assert eq8 + T * 2 * d * 4 == app + dec


def test_batch_decode_bytes_reduce_to_table6():
    kv, total = traffic.gqa_table(1024, 64, 64, 32, 8)
    assert traffic.batch_decode_bytes([1024], 32, 8, 64, 64) == total
    assert traffic.batch_partial_bytes([1024], 32, 8, 64, 64) == kv + 32 * 64 * 4
    assert traffic.batch_append_bytes(4, 8, 128, 128) == 4 * 8 * 256 * 4
