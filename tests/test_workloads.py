"""The seeded input generator: Philox4x32-10 known-answer vectors (the
published test vectors of Salmon et al. 2011), determinism across thread
counts and offsets, and the N(0,1) moments of its output."""
import numpy as np
import pytest

from paper_2607_19456_amd import workloads

KAT = [
    ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
    ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
    ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
     [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
]


@pytest.mark.parametrize("ctr,key,expect", KAT)
def test_philox_known_answers(ctr, key, expect):
    assert workloads.philox4x32_10(ctr, key) == expect


def test_same_bytes_for_any_thread_count_and_offset():
    a = workloads.normal(5, 9, (1000, 37), threads=1)
    b = workloads.normal(5, 9, (1000, 37), threads=7)
    assert np.array_equal(a, b)
    c = np.empty(1234, np.float32)
    workloads.fill_normal(c, 5, 9, offset=4321, threads=3)
    assert np.array_equal(c, a.reshape(-1)[4321:4321 + 1234])


def test_streams_and_seeds_differ():
    a = workloads.normal(0, 1, (4096,))
    assert not np.array_equal(a, workloads.normal(0, 2, (4096,)))
    assert not np.array_equal(a, workloads.normal(1, 1, (4096,)))


def test_standard_normal_moments():
    x = workloads.normal(0, 3, (1 << 20,)).astype(np.float64)
    assert abs(x.mean()) < 5e-3
    assert abs(x.std() - 1.0) < 5e-3
    assert abs((x ** 3).mean()) < 2e-2
    assert abs((x ** 4).mean() - 3.0) < 3e-2
    assert np.all(np.isfinite(x))


def test_cache_pads_rows_beyond_len_and_matches_flat_stream():
    lens = np.array([5, 0, 9], np.int32)
    K = workloads.cache(0, 2, lens, 2, 9, 4, np.nan)
    flat = workloads.normal(0, 2, (3, 2, 9, 4))
    for b in range(3):
        assert np.array_equal(K[b, :, :lens[b]], flat[b, :, :lens[b]])
        assert np.all(np.isnan(K[b, :, lens[b]:]))


def test_workload_table_is_consistent():
    for name, s in workloads.WORKLOADS.items():
        assert s.h_q % s.h_kv == 0
        assert s.len_hi + s.steps <= s.n_max, name
        assert 1 <= s.len_lo <= s.len_hi
    c5 = workloads.get("c5")
    lens = workloads.draw_lengths(c5)
    assert lens.min() >= 65536 and lens.max() <= 131072 - 64
