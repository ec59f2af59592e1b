"""Pins of the attention oracle (Eq. 2 and the shared-prefix form of Eq. 4).

Each check is independent of the oracle's own formula: brute-force loops in
plain Python, closed forms derived by hand, invariants of unmasked softmax
attention, and Lemma 1 of the appendix.
"""
import math

import numpy as np
import pytest

from oracle.attention import (attention, attention_weights, full_attention, kv_head_of,
                              shared_prefix_attention)


def _brute_force(q, keys, vals, scale):
    """Eq. 2 with explicit loops and math.exp (no max subtraction, no numpy)."""
    out = []
    for qi in q:
        logits = [scale * sum(a * b for a, b in zip(qi, kj)) for kj in keys]
        ws = [math.exp(x) for x in logits]
        z = sum(ws)
        out.append([sum(w * vj[c] for w, vj in zip(ws, vals)) / z for c in range(len(vals[0]))])
    return np.array(out)


def test_brute_force_tiny():
    rng = np.random.default_rng(0)
    B, H, m, n_s, dh = 1, 1, 3, 2, 4
    q = rng.normal(size=(B, H, n_s, dh))
    kp, vp = rng.normal(size=(H, m, dh)), rng.normal(size=(H, m, dh))
    ks, vs = rng.normal(size=(B, H, n_s, dh)), rng.normal(size=(B, H, n_s, dh))
    got = shared_prefix_attention(q, kp, vp, ks, vs, 0.5)
    keys = list(kp[0]) + list(ks[0, 0])
    vals = list(vp[0]) + list(vs[0, 0])
    ref = _brute_force(q[0, 0], keys, vals, 0.5)
    np.testing.assert_allclose(got[0, 0], ref, rtol=1e-13, atol=1e-13)


def test_brute_force_batched_gqa():
    """Two requests, Hq=4 over Hkv=2: each request sees only its own suffix."""
    rng = np.random.default_rng(1)
    B, Hq, Hkv, m, n_s, dh = 2, 4, 2, 3, 2, 4
    q = rng.normal(size=(B, Hq, n_s, dh))
    kp, vp = rng.normal(size=(Hkv, m, dh)), rng.normal(size=(Hkv, m, dh))
    ks, vs = rng.normal(size=(B, Hkv, n_s, dh)), rng.normal(size=(B, Hkv, n_s, dh))
    got = shared_prefix_attention(q, kp, vp, ks, vs, 0.3)
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)          # contiguous groups of Hq/Hkv heads
            ref = _brute_force(q[b, h], list(kp[g]) + list(ks[b, g]),
                               list(vp[g]) + list(vs[b, g]), 0.3)
            np.testing.assert_allclose(got[b, h], ref, rtol=1e-13, atol=1e-13)


def test_hand_derived_weights():
    """scale = ln 3, q = e0, keys e0 and e1: logits (ln 3, 0) so the weights are
    exactly (3/4, 1/4) and the output is 3/4 v0 + 1/4 v1."""
    q = np.array([[1.0, 0.0]])
    k = np.array([[1.0, 0.0], [0.0, 1.0]])
    v = np.array([[4.0, -8.0], [8.0, 4.0]])
    o = attention(q, k, v, math.log(3.0))
    np.testing.assert_allclose(o, [[5.0, -5.0]], rtol=0, atol=1e-14)


def test_closed_forms():
    rng = np.random.default_rng(2)
    n, dh = 7, 8
    v = rng.normal(size=(n, dh))
    # identical keys -> every weight 1/n -> mean of the value rows
    k_same = np.tile(rng.normal(size=(1, dh)), (n, 1))
    np.testing.assert_allclose(attention(rng.normal(size=(3, dh)), k_same, v, 1.0),
                               np.tile(v.mean(0), (3, 1)), atol=1e-13)
    # q = 0 -> all logits 0 -> mean of the value rows
    np.testing.assert_allclose(attention(np.zeros((2, dh)), rng.normal(size=(n, dh)), v, 1.0),
                               np.tile(v.mean(0), (2, 1)), atol=1e-13)
    # constant values -> the constant (weights sum to 1)
    c = np.full((n, dh), -2.5)
    np.testing.assert_allclose(attention(rng.normal(size=(4, dh)), rng.normal(size=(n, dh)), c, 1.0),
                               np.full((4, dh), -2.5), atol=1e-13)
    # one key 40 logits above the rest -> that key's value row (e^-40 ~ 4e-18)
    k = np.zeros((n, dh))
    k[3, 0] = 40.0
    q = np.zeros((1, dh))
    q[0, 0] = 1.0
    np.testing.assert_allclose(attention(q, k, v, 1.0), v[3:4], atol=1e-15 * n + 1e-16)


def test_rows_sum_to_one():
    rng = np.random.default_rng(3)
    w = attention_weights(rng.normal(size=(5, 16)) * 4, rng.normal(size=(9, 16)) * 4, 0.25)
    np.testing.assert_allclose(w.sum(1), 1.0, atol=1e-14)
    assert (w > 0).all()


def test_permutation_across_split():
    """Unmasked attention is invariant under a joint permutation of the K/V rows,
    including permutations that move rows between the prefix and the suffix."""
    rng = np.random.default_rng(4)
    B, H, m, n_s, dh = 2, 2, 5, 4, 8
    q = rng.normal(size=(B, H, n_s, dh))
    kp, vp = rng.normal(size=(H, m, dh)), rng.normal(size=(H, m, dh))
    ks, vs = rng.normal(size=(B, H, n_s, dh)), rng.normal(size=(B, H, n_s, dh))
    ref = shared_prefix_attention(q, kp, vp, ks, vs, 0.35)
    for b in range(B):
        for h in range(H):
            k_all = np.concatenate([kp[h], ks[b, h]])
            v_all = np.concatenate([vp[h], vs[b, h]])
            perm = rng.permutation(m + n_s)
            got = attention(q[b, h], k_all[perm], v_all[perm], 0.35)
            np.testing.assert_allclose(got, ref[b, h], atol=1e-13)
    # permuting query rows permutes the output rows
    perm = rng.permutation(n_s)
    got = shared_prefix_attention(q[:, :, perm], kp, vp, ks, vs, 0.35)
    np.testing.assert_allclose(got, ref[:, :, perm], atol=1e-13)


def test_fresh_prefix_reproduces_full_attention():
    """Supplying the prefix K/V of the same sequence as 'cache' gives exactly the
    full bidirectional attention of the suffix rows."""
    rng = np.random.default_rng(5)
    B, H, m, n_s, dh = 1, 3, 6, 5, 8
    k = rng.normal(size=(B, H, m + n_s, dh))
    v = rng.normal(size=(B, H, m + n_s, dh))
    q = rng.normal(size=(B, H, m + n_s, dh))
    full = full_attention(q, k, v, 0.4)
    split = shared_prefix_attention(q[:, :, m:], k[0, :, :m], v[0, :, :m], k[:, :, m:], v[:, :, m:], 0.4)
    np.testing.assert_allclose(split, full[:, :, m:], atol=1e-13)


def test_gqa_equals_expanded_mha():
    rng = np.random.default_rng(6)
    B, Hq, Hkv, m, n_s, dh = 2, 28, 4, 5, 3, 8
    q = rng.normal(size=(B, Hq, n_s, dh))
    kp, vp = rng.normal(size=(Hkv, m, dh)), rng.normal(size=(Hkv, m, dh))
    ks, vs = rng.normal(size=(B, Hkv, n_s, dh)), rng.normal(size=(B, Hkv, n_s, dh))
    got = shared_prefix_attention(q, kp, vp, ks, vs, 0.2)
    G = Hq // Hkv
    exp = shared_prefix_attention(q, np.repeat(kp, G, 0), np.repeat(vp, G, 0),
                                  np.repeat(ks, G, 1), np.repeat(vs, G, 1), 0.2)
    np.testing.assert_allclose(got, exp, atol=1e-14)
    assert [kv_head_of(h, 28, 4) for h in (0, 6, 7, 13, 14, 27)] == [0, 0, 1, 1, 2, 3]


@pytest.mark.parametrize("m", [1, 4, 9])
def test_lemma1_leakage_bound(m):
    """Lemma 1: ||Attn_i - renormalised-over-prefix Attn_i|| <= 2 B_V rho_i where
    rho_i is the attention mass on non-prefix keys and B_V bounds ||v_j||."""
    rng = np.random.default_rng(7 + m)
    n, dh = 12, 6
    q, k, v = rng.normal(size=(4, dh)) * 2, rng.normal(size=(n, dh)), rng.normal(size=(n, dh))
    w = attention_weights(q, k, 0.7)
    o = attention(q, k, v, 0.7)
    bv = np.linalg.norm(v, axis=1).max()
    for i in range(4):
        rho = w[i, m:].sum()
        tilde = (w[i, :m] / (1.0 - rho)) @ v[:m]
        assert np.linalg.norm(o[i] - tilde) <= 2 * bv * rho * (1 + 1e-12)
