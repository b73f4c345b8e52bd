"""The seeded operand generator: pinned to SplitMix64's published output and to
its own plain-Python definition (the bulk loops are compiled C)."""
import math

import numpy as np
import pytest

import seeded_inputs as S


def test_splitmix64_published_sequence():
    # SplitMix64 (Steele, Lea, Flood 2014) started from state 0: its first three
    # outputs.  Stream 0 of the counter-based form walks the same states.
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [int(v) for v in S.stream(0, 3)] == want
    assert [S.element(0, i) for i in range(3)] == want


@pytest.mark.parametrize("seed", [1, 1001, 4002, 2 ** 31 + 5])
def test_bulk_stream_matches_definition(seed):
    x = S.stream(seed, 5000, offset=123)
    for i in range(0, 5000, 97):
        assert int(x[i]) == S.element(seed, 123 + i)


@pytest.mark.parametrize("dist", ["uniform", "normal", "wide"])
def test_bulk_distributions_match_definition(dist):
    a = S.make(dist, 777, (37, 53), np.float64).ravel()
    for i in range(0, a.size, 11):
        assert a[i] == S.value(dist, 777, i)


def test_distribution_ranges():
    u = S.uniform(5, (100000,))
    assert u.min() >= -1.0 and u.max() < 1.0 and abs(u.mean()) < 0.01
    w = S.wide(6, (100000,))
    e = np.frexp(np.abs(w))[1] - 1
    assert e.min() == -20 and e.max() == 20
    n = S.normal(7, (200000,))
    assert abs(n.mean()) < 0.01 and abs(n.std() - 1.0) < 0.01
    f = S.make("normal", 7, (10, 10), np.float32)
    assert f.dtype == np.float32 and np.array_equal(f, S.normal(7, (10, 10)).astype(np.float32))


def test_scaled_rows():
    a = S.make("normal_scaled_rows", 9, (300, 40), np.float64)
    big = np.flatnonzero(np.abs(a).max(axis=1) > 2.0 ** 10)
    assert big.size == math.ceil(0.01 * 300)
    assert sorted(S.permutation(9 + 500, 300)) == list(range(300))
