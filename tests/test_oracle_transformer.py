"""Pins of the step oracle: building blocks against loops and closed forms, and
the step against the properties the paper fixes (d = 0 is "no caching",
layer-1 KVs are exact, fresh prefix K/V reproduce the full forward, requests
are independent)."""
import math

import numpy as np
import pytest

from oracle import transformer as T


def _cfg(**kw):
    c = dict(n_layers=3, hidden=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn=48,
             rms_eps=1e-5, rope_theta=10000.0)
    c.update(kw)
    return c


def _weights(cfg, rng, scale_out=1.0):
    h, F = cfg["hidden"], cfg["ffn"]
    Hq, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    out = []
    for _ in range(cfg["n_layers"]):
        out.append({
            "w_qkv": rng.normal(size=((Hq + 2 * Hkv) * dh, h)) / math.sqrt(h),
            "w_o": rng.normal(size=(h, Hq * dh)) / math.sqrt(Hq * dh) * scale_out,
            "w_gate_up": rng.normal(size=(2 * F, h)) / math.sqrt(h),
            "w_down": rng.normal(size=(h, F)) / math.sqrt(F) * scale_out,
            "attn_norm": 1 + 0.1 * rng.normal(size=h),
            "ffn_norm": 1 + 0.1 * rng.normal(size=h),
        })
    return out


# ---------------------------------------------------------------- blocks

def test_rmsnorm_constant_and_loop():
    g = np.array([0.5, 2.0, -1.0])
    c = -3.0
    y = T.rms_norm(np.full((1, 3), c), g, 1e-5)
    np.testing.assert_allclose(y[0], np.sign(c) * g * abs(c) / math.sqrt(c * c + 1e-5), rtol=1e-14)
    rng = np.random.default_rng(0)
    x, gg = rng.normal(size=(2, 5)), rng.normal(size=5)
    for r in range(2):
        ms = sum(t * t for t in x[r]) / 5
        ref = [x[r, i] / math.sqrt(ms + 1e-6) * gg[i] for i in range(5)]
        np.testing.assert_allclose(T.rms_norm(x, gg, 1e-6)[r], ref, rtol=1e-13)


def test_rope_two_dim_is_plane_rotation():
    """dh = 2: one pair with frequency theta^0 = 1, i.e. a rotation by pos radians."""
    x = np.array([[[0.3, -1.2], [0.3, -1.2], [2.0, 0.5]]])        # [H=1, n=3, 2]
    pos = np.array([0, 1, 7])
    y = T.rope(x, pos, 500000.0)
    for i, p in enumerate(pos):
        a, b = x[0, i]
        np.testing.assert_allclose(y[0, i], [a * math.cos(p) - b * math.sin(p),
                                             b * math.cos(p) + a * math.sin(p)], atol=1e-15)


def test_rope_pairs_and_frequencies():
    """dh = 8: dims i and i+4 rotate together at frequency theta^(-2i/8)."""
    theta = 100.0
    x = np.zeros((1, 1, 8))
    x[0, 0, 1] = 1.0                    # unit vector on the first coordinate of pair 1
    y = T.rope(x, np.array([3]), theta)
    a = 3 * theta ** (-2.0 / 8)
    exp = np.zeros(8)
    exp[1], exp[5] = math.cos(a), math.sin(a)
    np.testing.assert_allclose(y[0, 0], exp, atol=1e-15)


def test_rope_norm_and_relative_position():
    rng = np.random.default_rng(1)
    q, k = rng.normal(size=(2, 5, 16)), rng.normal(size=(2, 5, 16))
    p1, p2 = np.arange(5), np.array([9, 3, 0, 12, 4])
    qr = T.rope(q, p1, 500000.0)
    np.testing.assert_allclose(np.linalg.norm(qr, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-13)
    base = np.einsum("hid,hjd->hij", T.rope(q, p1, 1e4), T.rope(k, p2, 1e4))
    shifted = np.einsum("hid,hjd->hij", T.rope(q, p1 + 1000, 1e4), T.rope(k, p2 + 1000, 1e4))
    np.testing.assert_allclose(shifted, base, atol=1e-9)


def test_silu_values():
    np.testing.assert_allclose(T.silu(np.array([0.0, 30.0, -30.0, 1.0])),
                               [0.0, 30.0 / (1 + math.exp(-30.0)), -30.0 / (1 + math.exp(30.0)), 1 / (1 + math.exp(-1))],
                               rtol=1e-14, atol=1e-20)


def _layer_loops(x, lw, cfg, pos):
    """One full layer written with plain Python loops (independent of the oracle)."""
    n, h = len(x), cfg["hidden"]
    Hq, Hkv, dh, F = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"], cfg["ffn"]
    eps, th = cfg["rms_eps"], cfg["rope_theta"]

    def norm(row, g):
        r = math.sqrt(sum(t * t for t in row) / h + eps)
        return [row[i] / r * g[i] for i in range(h)]

    def matvec(W, a, r0, nr, bias=None):
        return [sum(W[r0 + r][c] * a[c] for c in range(len(a))) + (bias[r0 + r] if bias else 0.0)
                for r in range(nr)]

    def rot(vec, p):
        out = list(vec)
        for i in range(dh // 2):
            ang = p * th ** (-2.0 * i / dh)
            a, b = vec[i], vec[i + dh // 2]
            out[i] = a * math.cos(ang) - b * math.sin(ang)
            out[i + dh // 2] = b * math.cos(ang) + a * math.sin(ang)
        return out

    Q, K, V = [], [], []
    for t in range(n):
        a = norm(x[t], lw["attn_norm"])
        bq = lw.get("b_qkv")
        Q.append([rot(matvec(lw["w_qkv"], a, hd * dh, dh, bq), pos[t]) for hd in range(Hq)])
        K.append([rot(matvec(lw["w_qkv"], a, (Hq + g) * dh, dh, bq), pos[t]) for g in range(Hkv)])
        V.append([matvec(lw["w_qkv"], a, (Hq + Hkv + g) * dh, dh, bq) for g in range(Hkv)])
    out = []
    for t in range(n):
        o = []
        for hd in range(Hq):
            g = hd // (Hq // Hkv)
            lg = [sum(Q[t][hd][i] * K[j][g][i] for i in range(dh)) / math.sqrt(dh) for j in range(n)]
            mx = max(lg)
            w = [math.exp(v - mx) for v in lg]
            z = sum(w)
            o += [sum(w[j] * V[j][g][i] for j in range(n)) / z for i in range(dh)]
        xr = [x[t][i] + sum(lw["w_o"][i][c] * o[c] for c in range(Hq * dh)) for i in range(h)]
        f = norm(xr, lw["ffn_norm"])
        gate = matvec(lw["w_gate_up"], f, 0, F)
        up = matvec(lw["w_gate_up"], f, F, F)
        act = [gate[i] / (1 + math.exp(-gate[i])) * up[i] for i in range(F)]
        out.append([xr[i] + sum(lw["w_down"][i][c] * act[c] for c in range(F)) for i in range(h)])
    return np.array(out)


def test_layer_against_loops():
    cfg = _cfg(n_layers=1, hidden=8, n_heads=2, n_kv_heads=1, head_dim=4, ffn=6)
    rng = np.random.default_rng(2)
    lw = _weights(cfg, rng)[0]
    x = rng.normal(size=(3, 8))
    pos = np.array([5, 6, 7])
    got, _, _ = T.layer_full(x, lw, cfg, pos)
    lw_list = {k: v.tolist() for k, v in lw.items()}
    ref = _layer_loops(x.tolist(), lw_list, cfg, pos.tolist())
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_layer_with_qkv_bias_against_loops():
    """Q/K/V bias (Qwen2-style layers such as Dream-7B's): added to the
    projections before RoPE; GQA with a group of 3."""
    cfg = _cfg(n_layers=1, hidden=8, n_heads=3, n_kv_heads=1, head_dim=4, ffn=6)
    rng = np.random.default_rng(12)
    lw = _weights(cfg, rng)[0]
    lw["b_qkv"] = rng.normal(size=(5 * 4,))
    x = rng.normal(size=(3, 8))
    pos = np.array([2, 9, 4])
    got, _, _ = T.layer_full(x, lw, cfg, pos)
    lw_list = {k: v.tolist() for k, v in lw.items()}
    ref = _layer_loops(x.tolist(), lw_list, cfg, pos.tolist())
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    # the bias matters, and with zero weights the projections are the bias itself
    assert np.abs(got - T.layer_full(x, {**lw, "b_qkv": None}, cfg, pos)[0]).max() > 1e-6
    zero = {**lw, "w_qkv": np.zeros_like(lw["w_qkv"])}
    q, k, v = T.project_qkv(x, zero, cfg, pos)
    np.testing.assert_allclose(v[0], np.tile(lw["b_qkv"][16:20], (3, 1)), atol=1e-15)
    # position 0 leaves q unrotated
    q0, _, _ = T.project_qkv(x[:1], zero, cfg, np.array([0]))
    np.testing.assert_allclose(q0[:, 0], lw["b_qkv"][:12].reshape(3, 4), atol=1e-15)


# ---------------------------------------------------------------- step

@pytest.fixture(scope="module")
def setup():
    cfg = _cfg()
    rng = np.random.default_rng(3)
    layers = _weights(cfg, rng, scale_out=1 / math.sqrt(6))
    m, n_s, B = 7, 5, 3
    xp = rng.normal(size=(m, cfg["hidden"]))
    xs = rng.normal(size=(B, n_s, cfg["hidden"]))
    cache = T.populate(xp, layers, cfg, cfg["n_layers"])
    return cfg, layers, xp, xs, cache


def test_d0_is_no_caching(setup):
    cfg, layers, xp, xs, cache = setup
    got = T.step(cache, xs, 0, layers, cfg)
    for b in range(xs.shape[0]):
        full = T.full_forward(xp, xs[b], layers, cfg)
        np.testing.assert_allclose(got[b], full[xp.shape[0]:], atol=1e-12)


def test_fresh_cache_equals_full_forward_for_every_d(setup):
    cfg, layers, xp, xs, _ = setup
    m = xp.shape[0]
    for b in range(xs.shape[0]):
        rec = {}
        full = T.full_forward(xp, xs[b], layers, cfg, record=rec)
        fresh = T.cache_from_full_forward(rec, m, cfg["n_layers"], cfg)
        for d in range(cfg["n_layers"] + 1):
            got = T.step_one(fresh, xs[b], d, layers, cfg)
            np.testing.assert_allclose(got, full[m:], atol=1e-12)


def test_layer0_cache_is_exact(setup):
    """Footnote of Sec. 4.2: first-layer KVs come straight from the token's own
    input, so the cached layer-0 prefix K/V equal those of the full input."""
    cfg, layers, xp, xs, cache = setup
    m = xp.shape[0]
    rec = {}
    T.full_forward(xp, xs[1], layers, cfg, record=rec)
    np.testing.assert_allclose(cache["k"][0], rec["k"][0][:, :m], atol=1e-13)
    np.testing.assert_allclose(cache["v"][0], rec["v"][0][:, :m], atol=1e-13)
    # ... while deeper layers do differ (bidirectional attention mixes in the suffix)
    assert np.abs(cache["k"][1] - rec["k"][1][:, :m]).max() > 1e-6


def test_one_layer_model_d1_equals_d0():
    cfg = _cfg(n_layers=1)
    rng = np.random.default_rng(4)
    layers = _weights(cfg, rng)
    xp, xs = rng.normal(size=(6, 32)), rng.normal(size=(2, 4, 32))
    cache = T.populate(xp, layers, cfg, 1)
    np.testing.assert_allclose(T.step(cache, xs, 1, layers, cfg), T.step(cache, xs, 0, layers, cfg),
                               atol=1e-12)


def test_recomputed_kv_at_d_equal_cache(setup):
    """With the prefix residual re-entered from the cache at layer d, the prefix
    K/V recomputed by layer d equal the cached KV$_d."""
    cfg, layers, xp, xs, cache = setup
    for d in range(cfg["n_layers"]):
        rec = {}
        T.step_one(cache, xs[0], d, layers, cfg, record=rec)
        np.testing.assert_allclose(rec["deep_k"][d], cache["k"][d], atol=1e-12)
        np.testing.assert_allclose(rec["deep_v"][d], cache["v"][d], atol=1e-12)
        if d + 1 < cfg["n_layers"]:       # the next layer's prefix K/V see the suffix
            assert np.abs(rec["deep_k"][d + 1] - cache["k"][d + 1]).max() > 1e-6


def test_dL_is_suffix_only(setup):
    cfg, layers, xp, xs, cache = setup
    L = cfg["n_layers"]
    ref = T.step(cache, xs, L, layers, cfg)
    poisoned = dict(cache, h=np.full_like(cache["h"], np.nan))
    np.testing.assert_array_equal(T.step(poisoned, xs, L, layers, cfg), ref)
    other = dict(cache, k=cache["k"] * 1.5)
    assert np.abs(T.step(other, xs, L, layers, cfg) - ref).max() > 1e-6
    # at d < L the cached residual of layer d is used
    assert np.isnan(T.step(poisoned, xs, L - 1, layers, cfg)).all()


def test_requests_independent_and_permutable(setup):
    cfg, layers, xp, xs, cache = setup
    for d in (0, 1, 3):
        batch = T.step(cache, xs, d, layers, cfg)
        single = np.stack([T.step(cache, xs[b:b + 1], d, layers, cfg)[0] for b in range(len(xs))])
        np.testing.assert_allclose(batch, single, atol=1e-13)
        perm = [2, 0, 1]
        np.testing.assert_allclose(T.step(cache, xs[perm], d, layers, cfg), batch[perm], atol=1e-13)


def test_partial_populate_layout(setup):
    cfg, layers, xp, xs, cache = setup
    part = T.populate(xp, layers, cfg, 1)
    assert part["k"].shape[0] == 1 and part["h"].shape[0] == 2
    np.testing.assert_allclose(part["h"], cache["h"][:2], atol=1e-14)
    np.testing.assert_allclose(T.step(part, xs, 1, layers, cfg), T.step(cache, xs, 1, layers, cfg),
                               atol=1e-13)
    none = T.populate(xp, layers, cfg, 0)
    assert none["k"].shape[0] == 0 and none["h"].shape[0] == 1
    np.testing.assert_array_equal(none["h"][0], xp)


# ---------------------------------------------------------------- Eq. 5 reuse

def test_refresh_schedule_closed_forms():
    """Eq. 5: step 1 refreshes; with delta = 16 the refresh steps of a 128-step
    generation are 1, 17, ..., 113 (eight of them, ceil(T / delta) in general);
    delta = 1 refreshes at every step."""
    assert T.is_refresh_step(1, 16)
    assert [t for t in range(1, 129) if T.is_refresh_step(t, 16)] == [1 + 16 * i for i in range(8)]
    for delta in (1, 2, 3, 7, 16, 64):
        for n in (1, 5, 16, 17, 128):
            assert sum(T.is_refresh_step(t, delta) for t in range(1, n + 1)) == -(-n // delta)
    assert all(T.is_refresh_step(t, 1) for t in range(1, 50))
    # a refresh is followed by exactly delta - 1 reuse steps
    assert not any(T.is_refresh_step(t, 4) for t in (2, 3, 4)) and T.is_refresh_step(5, 4)


def test_reuse_right_after_refresh_is_exact(setup):
    """The suffix rows of a full layer attend over [prefix K/V ; suffix K/V], so
    feeding the refresh step's own prefix K/V back with the same suffix input
    reproduces the refresh output for every depth."""
    cfg, layers, xp, xs, cache = setup
    for d in range(cfg["n_layers"] + 1):
        for b in range(xs.shape[0]):
            rec = {}
            ref = T.step_one(cache, xs[b], d, layers, cfg, record=rec)
            got = T.step_reuse_one(cache, rec, xs[b], d, layers, cfg)
            np.testing.assert_allclose(got, ref, atol=1e-12)


def test_reuse_uses_own_deep_layers_only(setup):
    """Shallow layers read the shared cache, deep layers only the request's own
    record: poisoning the record below d changes nothing, poisoning it at any
    deep layer poisons the output, and another request's record is not
    interchangeable."""
    cfg, layers, xp, xs, cache = setup
    L = cfg["n_layers"]
    d = 1
    rec0, rec1 = {}, {}
    T.step_one(cache, xs[0], d, layers, cfg, record=rec0)
    T.step_one(cache, xs[1], d, layers, cfg, record=rec1)
    ref = T.step_reuse_one(cache, rec0, xs[2], d, layers, cfg)
    assert set(rec0["deep_k"]) == set(range(d, L))
    for l in range(d, L):
        bad = {"deep_k": dict(rec0["deep_k"]), "deep_v": dict(rec0["deep_v"])}
        bad["deep_v"][l] = np.full_like(bad["deep_v"][l], np.nan)
        assert np.isnan(T.step_reuse_one(cache, bad, xs[2], d, layers, cfg)).all()
    other = T.step_reuse_one(cache, rec1, xs[2], d, layers, cfg)
    assert np.abs(other - ref).max() > 1e-6
    # the stale prefix K/V make a reuse step differ from a fresh recompute
    assert np.abs(T.step_one(cache, xs[2], d, layers, cfg) - ref).max() > 1e-6
    # at d = L there are no deep layers and the record is never read
    np.testing.assert_array_equal(T.step_reuse_one(cache, {}, xs[2], L, layers, cfg),
                                  T.step_one(cache, xs[2], L, layers, cfg))


def test_first_layer_reuse_is_exact_for_any_suffix():
    """Footnote of Sec. 4.2: first-layer prefix K/V depend on the prefix tokens
    alone, so in a one-layer model with d = 0 reusing them across steps is
    exact whatever the new suffix."""
    cfg = _cfg(n_layers=1)
    rng = np.random.default_rng(6)
    layers = _weights(cfg, rng)
    xp, xs = rng.normal(size=(6, 32)), rng.normal(size=(2, 4, 32))
    cache = T.populate(xp, layers, cfg, 1)
    rec = {}
    T.step_one(cache, xs[0], 0, layers, cfg, record=rec)
    np.testing.assert_allclose(T.step_reuse_one(cache, rec, xs[1], 0, layers, cfg),
                               T.step_one(cache, xs[1], 0, layers, cfg), atol=1e-12)


def test_denoise_steps_schedule(setup):
    """delta = 1 is a refresh at every step (plain step per step); with delta = 3
    the refresh steps 1 and 4 match a fresh step of their own input whatever
    came before, and the reuse steps 2, 3, 5 depend on the inputs of their
    last refresh step but not on those of earlier reuse steps."""
    cfg, layers, xp, xs, cache = setup
    rng = np.random.default_rng(7)
    n_steps, d = 5, 1
    xsteps = xs[None] + 0.3 * rng.normal(size=(n_steps,) + xs.shape)
    every = T.denoise_steps(cache, xsteps, d, 1, layers, cfg)
    for t in range(n_steps):
        np.testing.assert_allclose(every[t], T.step(cache, xsteps[t], d, layers, cfg), atol=1e-12)
    base = T.denoise_steps(cache, xsteps, d, 3, layers, cfg)
    for t in (0, 3):
        np.testing.assert_allclose(base[t], every[t], atol=1e-12)
    for t in (1, 2, 4):
        assert np.abs(base[t] - every[t]).max() > 1e-6
    # changing the input of reuse step 2 changes step 2 only
    x2 = xsteps.copy()
    x2[1] += 1.0
    alt = T.denoise_steps(cache, x2, d, 3, layers, cfg)
    assert np.abs(alt[1] - base[1]).max() > 1e-6
    for t in (0, 2, 3, 4):
        np.testing.assert_array_equal(alt[t], base[t])
    # changing the input of refresh step 1 changes every step up to step 4
    x1 = xsteps.copy()
    x1[0] += 1.0
    alt = T.denoise_steps(cache, x1, d, 3, layers, cfg)
    for t in (0, 1, 2):
        assert np.abs(alt[t] - base[t]).max() > 1e-6
    for t in (3, 4):
        np.testing.assert_array_equal(alt[t], base[t])
    # requests stay independent across the whole sequence
    one = T.denoise_steps(cache, xsteps[:, 1:2], d, 3, layers, cfg)
    np.testing.assert_allclose(one[:, 0], base[:, 1], atol=1e-13)


# ---------------------------------------------------------------- several prefixes

def test_multi_prefix_d0_is_each_requests_full_forward():
    """d = 0 is no caching (Sec. 3.1): with several prefixes of different
    lengths in one batch, every request equals the un-cached forward of its own
    (prefix, suffix), whatever the other groups hold."""
    cfg = _cfg()
    rng = np.random.default_rng(8)
    layers = _weights(cfg, rng, scale_out=1 / math.sqrt(6))
    prefixes = [rng.normal(size=(m, cfg["hidden"])) for m in (7, 3, 10)]
    counts = [2, 1, 3]
    xs = rng.normal(size=(sum(counts), 4, cfg["hidden"]))
    caches = [T.populate(p, layers, cfg, cfg["n_layers"]) for p in prefixes]
    got = T.step_multi(caches, counts, xs, 0, layers, cfg)
    owner = [g for g, c in enumerate(counts) for _ in range(c)]
    for b, g in enumerate(owner):
        full = T.full_forward(prefixes[g], xs[b], layers, cfg)
        np.testing.assert_allclose(got[b], full[len(prefixes[g]):], atol=1e-12)


def test_multi_prefix_groups_are_independent_and_use_their_own_prefix():
    cfg = _cfg()
    rng = np.random.default_rng(9)
    layers = _weights(cfg, rng, scale_out=1 / math.sqrt(6))
    pa, pb = rng.normal(size=(6, cfg["hidden"])), rng.normal(size=(9, cfg["hidden"]))
    ca = T.populate(pa, layers, cfg, cfg["n_layers"])
    cb = T.populate(pb, layers, cfg, cfg["n_layers"])
    xs = rng.normal(size=(3, 5, cfg["hidden"]))
    for d in (1, 3):
        both = T.step_multi([ca, cb], [1, 2], xs, d, layers, cfg)
        np.testing.assert_allclose(both[:1], T.step(ca, xs[:1], d, layers, cfg), atol=1e-13)
        np.testing.assert_allclose(both[1:], T.step(cb, xs[1:], d, layers, cfg), atol=1e-13)
        # the same requests over the other prefix give other outputs
        swapped = T.step_multi([cb, ca], [1, 2], xs, d, layers, cfg)
        assert np.abs(swapped - both).max() > 1e-6
        # one group of one prefix is the single-prefix step
        np.testing.assert_allclose(T.step_multi([ca], [3], xs, d, layers, cfg),
                                   T.step(ca, xs, d, layers, cfg), atol=1e-13)
