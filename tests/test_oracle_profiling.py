"""Pins of the profiling oracle: the cosine against values fixed by geometry
and against Lemma 3's identity (App. B), first-layer similarity 1 (footnote
of Sec. 4.2), the b rule and table T on hand-made cases."""
import math

import numpy as np
import pytest

from oracle import profiling as P
from tests.test_oracle_transformer import _cfg, _weights


def test_cosine_fixed_values():
    assert P.kv_similarity([1.0, 0.0], [1.0, 1.0]) == pytest.approx(1 / math.sqrt(2), abs=1e-15)
    a = np.array([[3.0, -1.0], [2.0, 5.0]])
    assert P.kv_similarity(a, a) == pytest.approx(1.0, abs=1e-15)
    assert P.kv_similarity(a, -2.5 * a) == pytest.approx(-1.0, abs=1e-15)
    assert P.kv_similarity([1.0, 2.0, 0.0], [-2.0, 1.0, 7.0]) == pytest.approx(0.0, abs=1e-15)
    # flattening: the layout of the two operands must agree, not their shape's meaning
    rng = np.random.default_rng(0)
    x, y = rng.normal(size=(2, 3, 4, 5)), rng.normal(size=(2, 3, 4, 5))
    assert P.kv_similarity(x, y) == pytest.approx(P.kv_similarity(x.ravel(), y.ravel()), abs=1e-15)
    assert P.kv_similarity(x, y) == pytest.approx(P.kv_similarity(7 * x, 0.1 * y), abs=1e-14)
    with pytest.raises(AssertionError):
        P.kv_similarity(np.zeros(3), np.ones(3))


def test_lemma3_identity_and_bound():
    """App. B, Lemma 3: 1 - cos(a, b) = (|a-b|^2 - (|a|-|b|)^2) / (2|a||b|)
    <= |a-b|^2 / (2|a||b|), for any nonzero a, b."""
    rng = np.random.default_rng(1)
    for n in (2, 17, 1000):
        for scale in (1e-3, 1.0, 50.0):
            a = rng.normal(size=n)
            b = a + scale * rng.normal(size=n)
            na, nb, dd = np.linalg.norm(a), np.linalg.norm(b), np.linalg.norm(a - b)
            one_minus = 1 - P.kv_similarity(a, b)
            ident = (dd ** 2 - (na - nb) ** 2) / (2 * na * nb)
            assert one_minus == pytest.approx(ident, rel=1e-7, abs=1e-13)
            assert one_minus <= dd ** 2 / (2 * na * nb) + 1e-15


def test_first_layer_similarity_is_one_and_deeper_below():
    """Footnote of Sec. 4.2: first-layer KVs come from the tokens' own inputs,
    so sim_1 = 1 and b >= 1 for any tau <= 1; deeper layers see the suffix."""
    cfg = _cfg(n_layers=4)
    rng = np.random.default_rng(2)
    layers = _weights(cfg, rng, scale_out=1 / math.sqrt(8))
    xp, xs = rng.normal(size=(9, cfg["hidden"])), rng.normal(size=(4, cfg["hidden"]))
    sims = P.profile_request(xp, xs, layers, cfg)
    assert sims.shape == (4,)
    assert sims[0] == pytest.approx(1.0, abs=1e-12)
    assert (sims[1:] < 1 - 1e-9).all() and (sims > -1).all()
    assert P.shallow_depth(sims, 1.0 - 1e-9) >= 1


def test_longer_prefix_raises_similarity():
    """Sec. 4.2: the larger the shared-prefix ratio, the less the suffix moves
    the prefix KVs.  With the suffix fixed, a prefix 20x longer (the extra
    tokens prepended) leaves the second layer's similarity higher."""
    cfg = _cfg(n_layers=2)
    rng = np.random.default_rng(3)
    layers = _weights(cfg, rng)
    tail = rng.normal(size=(4, cfg["hidden"]))
    xs = rng.normal(size=(8, cfg["hidden"]))
    long_p = np.concatenate([rng.normal(size=(76, cfg["hidden"])), tail])
    s_short = P.profile_request(tail, xs, layers, cfg)[1]
    s_long = P.profile_request(long_p, xs, layers, cfg)[1]
    assert s_long > s_short


def test_shallow_depth_rule():
    tau = 0.97
    assert P.shallow_depth([1.0, 0.98, 0.96, 0.99], tau) == 2     # stops at the first miss
    assert P.shallow_depth([1.0, 0.97, 0.975], tau) == 3          # >= tau counts
    assert P.shallow_depth([0.5, 0.99], tau) == 0
    assert P.shallow_depth([], tau) == 0


def test_table_floor_mean_and_lookup():
    ratios = [0.5, 0.5, 0.5, 0.75, 0.75, 1.0]
    depths = [3, 4, 4, 10, 11, 32]
    T = P.build_table(ratios, depths, n_buckets=4)
    # buckets 1..4 = r 0.25, 0.5, 0.75, 1.0: floor(11/3) = 3, floor(21/2) = 10, 32
    assert T == [-1, -1, 3, 10, 32]
    assert P.lookup_depth(T, 0.5) == 3
    assert P.lookup_depth(T, 0.74) == 3       # rounds down to the 0.5 bucket
    assert P.lookup_depth(T, 0.75) == 10
    assert P.lookup_depth(T, 0.99) == 10
    assert P.lookup_depth(T, 1.0) == 32
    assert P.lookup_depth(T, 0.3) == 0        # nothing at or below
    assert P.shared_prefix_ratio(1536, 512) == 0.75
    with pytest.raises(AssertionError):
        P.build_table([0.333], [1], n_buckets=4)
