"""Oracle: bidirectional attention (Sec. 2.2, Eq. 2) in float64.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Eq. 2 defines the attention output of a query as the softmax-weighted sum of
the value vectors of *all* n tokens of the input string, with weights
softmax_j(q . k_j / sqrt(d_k)).  There is no causal mask: every query sees
every key.  The shallow layers of BiCache (Eq. 4) attend over the cached
prefix KVs followed by the request's own suffix KVs, which is the same
definition applied to the concatenated key/value sequence.
"""
import numpy as np


def attention_weights(q, k, scale):
    """Softmax weights of Eq. 2 for one head.

    q: [n_q, d_k], k: [n_k, d_k] (float64).  Returns W [n_q, n_k] whose row i
    is softmax_j(scale * q_i . k_j).  Subtracting the row maximum before
    exponentiating does not change the result (softmax is shift invariant)
    and keeps exp() finite.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    logits = (q @ k.T) * scale
    logits = logits - logits.max(axis=1, keepdims=True)
    e = np.exp(logits)
    return e / e.sum(axis=1, keepdims=True)


def attention(q, k, v, scale):
    """Eq. 2 for one head: o_i = sum_j softmax_j(scale q_i . k_j) v_j.

    q: [n_q, d_k], k: [n_k, d_k], v: [n_k, d_v].  Returns [n_q, d_v] float64.
    """
    w = attention_weights(q, k, scale)
    return w @ np.asarray(v, dtype=np.float64)


def kv_head_of(h, n_q_heads, n_kv_heads):
    """Grouped-query mapping: query head h reads KV head floor(h*Hkv/Hq).

    With Hq a multiple of Hkv this puts consecutive runs of Hq/Hkv query heads
    on one KV head (contiguous groups); with Hq == Hkv it is the identity.
    """
    return (h * n_kv_heads) // n_q_heads


def shared_prefix_attention(q, k_pre, v_pre, k_suf, v_suf, scale):
    """Shallow-layer attention of Eq. 4: suffix queries over [cached prefix ; own suffix].

    q:      [B, Hq, n_s, dh]   suffix queries of each request
    k_pre:  [Hkv, m, dh]       ONE shared copy of the cached prefix keys
    v_pre:  [Hkv, m, dh]       ... and values
    k_suf:  [B, Hkv, n_s, dh]  each request's own suffix keys
    v_suf:  [B, Hkv, n_s, dh]  ... and values
    Returns [B, Hq, n_s, dh] float64.

    Request b attends to the shared prefix and to its own suffix only; there is
    no attention between different requests (each request is its own input
    string (p, z_t)).
    """
    q = np.asarray(q, dtype=np.float64)
    B, Hq, n_s, dh = q.shape
    Hkv = k_pre.shape[0]
    out = np.empty((B, Hq, n_s, v_pre.shape[-1]), dtype=np.float64)
    for b in range(B):
        for h in range(Hq):
            g = kv_head_of(h, Hq, Hkv)
            k_all = np.concatenate([np.asarray(k_pre[g], np.float64),
                                    np.asarray(k_suf[b, g], np.float64)], axis=0)
            v_all = np.concatenate([np.asarray(v_pre[g], np.float64),
                                    np.asarray(v_suf[b, g], np.float64)], axis=0)
            out[b, h] = attention(q[b, h], k_all, v_all, scale)
    return out


def full_attention(q, k, v, scale):
    """Bidirectional attention of every request over its own whole sequence.

    q: [B, Hq, n, dh], k, v: [B, Hkv, n, dh].  Returns [B, Hq, n, dh] float64.
    This is the deep-layer attention (no shared segment).
    """
    q = np.asarray(q, dtype=np.float64)
    B, Hq, n, dh = q.shape
    Hkv = k.shape[1]
    out = np.empty((B, Hq, n, v.shape[-1]), dtype=np.float64)
    for b in range(B):
        for h in range(Hq):
            g = kv_head_of(h, Hq, Hkv)
            out[b, h] = attention(q[b, h], k[b, g], v[b, g], scale)
    return out
