"""Pins of the host-side oracle pieces: XXH64 (prefix key) and the FIFO store."""
import numpy as np
import pytest
import xxhash

from oracle.cache_table import FifoTable
from oracle.xxh64 import prefix_key, xxh64


def test_xxh64_empty_known_answer():
    # The published XXH64 of the empty input with seed 0.
    assert xxh64(b"", 0) == 0xEF46DB3751D8E999


@pytest.mark.parametrize("n", list(range(0, 70)) + [100, 1000, 4099])
def test_xxh64_matches_library(n):
    rng = np.random.default_rng(n)
    data = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
    for seed in (0, 1, 2**63 + 5):
        assert xxh64(data, seed) == xxhash.xxh64_intdigest(data, seed=seed)


def test_prefix_key_is_le_int32():
    ids = np.array([1, 2, 3, -7, 2**31 - 1, 128000], dtype=np.int64)
    assert prefix_key(ids) == xxhash.xxh64_intdigest(ids.astype("<i4").tobytes(), seed=0)


def test_fifo_table():
    t = FifoTable(2)
    assert t.insert(10, "a") is None
    assert t.insert(20, "b") is None
    assert t.insert(30, "c") == 10
    assert t.order() == [20, 30]
    with pytest.raises(KeyError):
        t.insert(20, "again")
    assert t.invalidate(20) and not t.invalidate(20)
    assert t.insert(40, "d") is None
    assert t.insert(50, "e") == 30
    assert t.order() == [40, 50] and t.lookup(40) == "d" and t.lookup(30) is None
