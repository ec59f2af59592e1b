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


def _single_part_cos(xp, xs, layers, cfg, l, part):
    """cos of one part (K or V) of layer l: cached prefix-only KVs against the
    prefix rows of the un-cached forward."""
    from oracle import transformer as TR
    m = xp.shape[0]
    cache = TR.populate(xp, layers, cfg, cfg["n_layers"])
    rec = {}
    TR.full_forward(xp, xs, layers, cfg, record=rec)
    a = cache[part][l].ravel()
    b = rec[part][l][:, :m].ravel()
    return float(a @ b) / (np.linalg.norm(a) * np.linalg.norm(b))


def test_kv_similarity_flattens_k_and_v_jointly():
    """Footnote of Sec. 4.1: K and V of a layer form ONE flattened vector.  With
    the layer's value projection zeroed its V part is 0, and the joint cosine
    must equal the cosine of the K parts alone; with the key projection zeroed,
    that of the V parts alone.  A K-only, V-only or averaged reading fails one
    of the two (and on the untouched model all three readings differ)."""
    cfg = _cfg(n_layers=3)
    rng = np.random.default_rng(11)
    layers = _weights(cfg, rng, scale_out=1 / math.sqrt(6))
    xp, xs = rng.normal(size=(10, cfg["hidden"])), rng.normal(size=(5, cfg["hidden"]))
    Hq, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    k_rows = slice(Hq * dh, (Hq + Hkv) * dh)
    v_rows = slice((Hq + Hkv) * dh, (Hq + 2 * Hkv) * dh)
    l = 1
    base = P.profile_request(xp, xs, layers, cfg)[l]
    ck = _single_part_cos(xp, xs, layers, cfg, l, "k")
    cv = _single_part_cos(xp, xs, layers, cfg, l, "v")
    assert min(abs(base - ck), abs(base - cv), abs(base - (ck + cv) / 2)) > 1e-6
    for zero, keep, part in ((v_rows, k_rows, "k"), (k_rows, v_rows, "v")):
        lz = [dict(lw) for lw in layers]
        w = lz[l]["w_qkv"].copy()
        w[zero] = 0.0
        lz[l]["w_qkv"] = w
        sim = P.profile_request(xp, xs, lz, cfg)[l]
        assert sim == pytest.approx(_single_part_cos(xp, xs, lz, cfg, l, part), abs=1e-12)
        assert sim < 1 - 1e-9
