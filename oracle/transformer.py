"""Oracle: one denoising-step forward of a DLM transformer, with BiCache's split.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

What is computed (all in float64, on inputs that are the same bf16 values the
GPU receives, widened exactly):

* A layer is pre-norm: a = RMSNorm(x) g_attn; q, k, v = a W_q^T, a W_k^T,
  a W_v^T (Eq. 1, projections of the layer's hidden state); rotary position
  embedding on q and k; bidirectional attention (Eq. 2); x += o W_o^T;
  f = RMSNorm(x) g_ffn; x += (silu(f W_g^T) * (f W_u^T)) W_d^T.  The paper
  does not spell out the layer; this LLaMA-style block (RMSNorm, rotate-half
  RoPE, SwiGLU, no biases) is the reading used throughout.
* populate: the prefix-only forward x_pref = p ("on a miss, compute the KVs
  of p at the first step for all layers and store them in H[k]", Sec. 5.2).
  It records the post-RoPE prefix K/V of every cached layer (the KV$ of
  Eq. 4) and the prefix residual entering each layer.
* step(d): layers l < d reuse the cached prefix K/V and project only the
  suffix rows (Eq. 4); layers l >= d recompute the prefix from the current
  request and run full bidirectional attention (refresh case of Eq. 5).
  d is the paper's b (its layers are 1-based, l <= b; here 0-based, l < d).
* step_reuse_one / denoise_steps: the steps between refreshes (second case
  of Eq. 5, refresh every delta steps, (t - 1) mod delta == 0): every layer
  is suffix-only, the deep layers attending over the prefix K/V that the
  request's last refresh step computed.
* step_multi: a batch over several cached prefixes (groups of consecutive
  requests, each group with its own cache).
* full_forward: the un-cached forward of (p, z_t) ("no caching"), which is
  what d = 0 must equal.

Reading of a point the paper leaves open: the shallow layers never process
the prefix rows, so the prefix hidden state that enters the first deep layer
is taken to be the prefix-only residual cached by populate.  A consequence
that the tests check: the prefix K/V recomputed at layer d equal the cached
KV$_d exactly.
"""
import os

import numpy as np

from .attention import attention, kv_head_of


# --------------------------------------------------------------------------
# building blocks
# --------------------------------------------------------------------------

def rms_norm(x, gain, eps):
    """y = x / sqrt(mean(x^2) + eps) * gain, row-wise over the hidden dim."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def rope_angles(positions, head_dim, theta):
    """Rotation angle pos * theta^(-2i/dh) for pair i = 0..dh/2-1.

    Returns [n, dh/2] float64.
    """
    half = head_dim // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    return np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]


def rope(x, positions, theta):
    """Rotate-half rotary embedding.

    x: [H, n, dh].  Dimension i is paired with i + dh/2 and the pair is rotated
    by the angle of its position:
        x'[i]      = x[i] cos(a) - x[i+dh/2] sin(a)
        x'[i+dh/2] = x[i+dh/2] cos(a) + x[i] sin(a)
    """
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    ang = rope_angles(positions, dh, theta)          # [n, half]
    c, s = np.cos(ang)[None], np.sin(ang)[None]       # [1, n, half]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x):
    """silu(x) = x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def project_qkv(x_res, lw, cfg, positions):
    """RMSNorm, then the Q/K/V projections (Eq. 1), then RoPE on q and k.

    x_res: [n, h] residual rows.  w_qkv rows are [Hq*dh query | Hkv*dh key |
    Hkv*dh value], each block head-major.  An optional bias lw["b_qkv"] (same
    row order; the Q/K/V bias of Qwen2-style models such as Dream-7B) is added
    to the projections before RoPE.  Returns q [Hq, n, dh], k [Hkv, n, dh],
    v [Hkv, n, dh].
    """
    Hq, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    n = x_res.shape[0]
    a = rms_norm(x_res, lw["attn_norm"], cfg["rms_eps"])
    proj = a @ lw["w_qkv"].T
    if lw.get("b_qkv") is not None:
        proj = proj + lw["b_qkv"]
    q = proj[:, : Hq * dh].reshape(n, Hq, dh).transpose(1, 0, 2)
    k = proj[:, Hq * dh: (Hq + Hkv) * dh].reshape(n, Hkv, dh).transpose(1, 0, 2)
    v = proj[:, (Hq + Hkv) * dh:].reshape(n, Hkv, dh).transpose(1, 0, 2)
    q = rope(q, positions, cfg["rope_theta"])
    k = rope(k, positions, cfg["rope_theta"])
    return q, k, v


def _workers():
    """Host threads the oracle may use (OMP_NUM_THREADS when set)."""
    try:
        n = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        n = 0
    return max(1, n or (os.cpu_count() or 1))


def attend(q, k_all, v_all, cfg):
    """Attention of every query head over the given K/V (no mask, Eq. 2).

    q: [Hq, n_q, dh]; k_all, v_all: [Hkv, n_k, dh].  Returns the attention
    output laid out token-major [n_q, Hq*dh] (head h occupies columns
    h*dh .. h*dh+dh-1), which is the input of the output projection.

    Heads are independent (each is Eq. 2 on its own Q/K/V), so large ones run
    on a pool of host threads, one head per task with single-threaded BLAS;
    every head's arithmetic is the same as in a serial loop.
    """
    Hq, n_q, dh = q.shape
    Hkv = k_all.shape[0]
    scale = 1.0 / np.sqrt(dh)

    def one_head(h):
        g = kv_head_of(h, Hq, Hkv)
        return attention(q[h], k_all[g], v_all[g], scale)

    workers = min(Hq, _workers())
    if workers > 1 and n_q * k_all.shape[1] >= (1 << 20):
        from concurrent.futures import ThreadPoolExecutor
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1, user_api="blas"), ThreadPoolExecutor(workers) as ex:
            heads = list(ex.map(one_head, range(Hq)))
    else:
        heads = [one_head(h) for h in range(Hq)]
    o = np.stack(heads)
    return o.transpose(1, 0, 2).reshape(n_q, Hq * dh)


def post_attention(x_res, o, lw, cfg):
    """x += o W_o^T; then x += (silu(f W_g^T) * f W_u^T) W_d^T with f = RMSNorm(x) g_ffn."""
    F = cfg["ffn"]
    x = x_res + o @ lw["w_o"].T
    f = rms_norm(x, lw["ffn_norm"], cfg["rms_eps"])
    gate = f @ lw["w_gate_up"][:F].T
    up = f @ lw["w_gate_up"][F:].T
    return x + (silu(gate) * up) @ lw["w_down"].T


def layer_full(x_res, lw, cfg, positions):
    """One layer over a whole sequence (every row projected, full attention).

    Returns (new residual [n, h], k [Hkv, n, dh], v [Hkv, n, dh]).
    """
    q, k, v = project_qkv(x_res, lw, cfg, positions)
    o = attend(q, k, v, cfg)
    return post_attention(x_res, o, lw, cfg), k, v


def layer_suffix(s_res, lw, cfg, k_pre, v_pre, positions):
    """One shallow layer (Eq. 4): only the suffix rows are projected; they
    attend over [cached prefix K/V ; own suffix K/V].

    s_res: [n_s, h]; k_pre, v_pre: [Hkv, m, dh] (the cached KV$ of this layer).
    Returns (new suffix residual, suffix k, suffix v).
    """
    q, k, v = project_qkv(s_res, lw, cfg, positions)
    k_all = np.concatenate([k_pre, k], axis=1)
    v_all = np.concatenate([v_pre, v], axis=1)
    o = attend(q, k_all, v_all, cfg)
    return post_attention(s_res, o, lw, cfg), k, v


# --------------------------------------------------------------------------
# populate / step / full forward
# --------------------------------------------------------------------------

def populate(x_prefix, layers, cfg, n_layers_to_cache):
    """Prefix-only forward (x_pref = p) over the first n_layers_to_cache layers.

    Returns a dict with
      "k", "v": [Lc, Hkv, m, dh]  post-RoPE prefix K/V of layers 0..Lc-1 (KV$)
      "h":      [nH, m, h]        prefix residual entering layers 0..nH-1,
                                  nH = min(Lc + 1, L)
      "m":      m
    Positions of the prefix are 0..m-1.
    """
    L = cfg["n_layers"]
    Lc = n_layers_to_cache
    assert 0 <= Lc <= L
    x = np.asarray(x_prefix, dtype=np.float64)
    m = x.shape[0]
    pos = np.arange(m)
    ks, vs, hs = [], [], []
    n_h = min(Lc + 1, L)
    for l in range(max(Lc, n_h)):
        if l < n_h:
            hs.append(x.copy())
        if l < Lc:
            x, k, v = layer_full(x, layers[l], cfg, pos)
            ks.append(k)
            vs.append(v)
    Hkv, dh = cfg["n_kv_heads"], cfg["head_dim"]
    empty_kv = np.zeros((0, Hkv, m, dh))
    return {
        "k": np.stack(ks) if ks else empty_kv,
        "v": np.stack(vs) if vs else empty_kv.copy(),
        "h": np.stack(hs) if hs else np.zeros((0, m, cfg["hidden"])),
        "m": m,
    }


def step_one(cache, s0, d, layers, cfg, record=None):
    """Step forward of ONE request at reuse depth d.

    s0: [n_s, h] suffix input rows.  Layers 0..d-1 reuse cache["k"/"v"][l]
    (Eq. 4); at layer d the prefix rows are re-entered from cache["h"][d] and
    layers d..L-1 run in full over all N = m + n_s rows (refresh case of
    Eq. 5).  Returns the final residual of the suffix rows [n_s, h].
    If ``record`` is a dict, the prefix-row K/V computed by deep layers are
    stored in it (record["deep_k"][l], record["deep_v"][l]).
    """
    L = cfg["n_layers"]
    m = cache["m"]
    s = np.asarray(s0, dtype=np.float64)
    n_s = s.shape[0]
    suf_pos = m + np.arange(n_s)
    for l in range(d):
        s, _, _ = layer_suffix(s, layers[l], cfg, cache["k"][l], cache["v"][l], suf_pos)
    if d == L:
        return s
    x = np.concatenate([cache["h"][d], s], axis=0)
    pos = np.arange(m + n_s)
    for l in range(d, L):
        x, k, v = layer_full(x, layers[l], cfg, pos)
        if record is not None:
            record.setdefault("deep_k", {})[l] = k[:, :m]
            record.setdefault("deep_v", {})[l] = v[:, :m]
    return x[m:]


def is_refresh_step(t, delta):
    """Eq. 5: step t (1-based) recomputes the deep layers' prefix KVs when
    (t - 1) mod delta == 0; otherwise they are reused from the previous step."""
    assert t >= 1 and delta >= 1
    return (t - 1) % delta == 0


def step_reuse_one(cache, deep, s0, d, layers, cfg):
    """A non-refresh step of ONE request (Eq. 4 for l < d, the second case of
    Eq. 5 for l >= d): every layer is suffix-only.  Shallow layers attend over
    the shared cache["k"/"v"][l]; deep layers over the request's own prefix
    K/V of its last refresh step, deep["deep_k"][l] / deep["deep_v"][l]
    ([Hkv, m, dh], as recorded by step_one).  Returns the suffix rows' final
    residual [n_s, h]."""
    L = cfg["n_layers"]
    m = cache["m"]
    s = np.asarray(s0, dtype=np.float64)
    suf_pos = m + np.arange(s.shape[0])
    for l in range(L):
        if l < d:
            kp, vp = cache["k"][l], cache["v"][l]
        else:
            kp, vp = deep["deep_k"][l], deep["deep_v"][l]
        s, _, _ = layer_suffix(s, layers[l], cfg, kp, vp, suf_pos)
    return s


def denoise_steps(cache, x_suffix_steps, d, delta, layers, cfg):
    """Steps t = 1..T of a batch under Eq. 4/5 with refresh interval delta.

    x_suffix_steps: [T, B, n_s, h], the suffix input of every step.  Refresh
    steps run step_one (deep layers recompute the prefix from the cached
    prefix-only residual) and record each request's deep prefix K/V; the
    other steps run step_reuse_one with the latest record.  Returns
    [T, B, n_s, h]."""
    T, B = x_suffix_steps.shape[0], x_suffix_steps.shape[1]
    deep = [None] * B
    out = []
    for t in range(1, T + 1):
        xs = x_suffix_steps[t - 1]
        row = []
        for b in range(B):
            if is_refresh_step(t, delta):
                rec = {}
                row.append(step_one(cache, xs[b], d, layers, cfg, record=rec))
                deep[b] = rec
            else:
                row.append(step_reuse_one(cache, deep[b], xs[b], d, layers, cfg))
        out.append(np.stack(row))
    return np.stack(out)


def step(cache, x_suffix, d, layers, cfg, requests=None):
    """Step forward of a batch: every request independently (requests do not
    attend to each other).  x_suffix: [B, n_s, h].  Returns [B', n_s, h] for
    the requested subset (all requests by default)."""
    L = cfg["n_layers"]
    assert 0 <= d <= L
    idx = range(x_suffix.shape[0]) if requests is None else requests
    return np.stack([step_one(cache, x_suffix[b], d, layers, cfg) for b in idx])


def step_multi(caches, counts, x_suffix, d, layers, cfg):
    """Step of a batch whose requests use several cached prefixes (the
    multi-tenant setting of Sec. 6.5; each request's prefix is looked up in H,
    Sec. 5.2): group g is counts[g] consecutive requests of x_suffix
    [B, n_s, h] over caches[g].  Every request is step_one over its own
    group's cache.  Returns [B, n_s, h]."""
    assert len(caches) == len(counts) and sum(counts) == len(x_suffix)
    out, i = [], 0
    for cache, cnt in zip(caches, counts):
        for _ in range(cnt):
            out.append(step_one(cache, x_suffix[i], d, layers, cfg))
            i += 1
    return np.stack(out)


def full_forward(x_prefix, x_suffix_one, layers, cfg, record=None):
    """Un-cached ("no caching") forward of the input string (p, z).

    x_prefix: [m, h]; x_suffix_one: [n_s, h].  Returns the final residual of
    all N rows [N, h].  If ``record`` is a dict it receives, per layer, the
    residual entering the layer ("h") and the post-RoPE K/V ("k", "v"), all
    rows.
    """
    x = np.concatenate([np.asarray(x_prefix, np.float64),
                        np.asarray(x_suffix_one, np.float64)], axis=0)
    pos = np.arange(x.shape[0])
    for l in range(cfg["n_layers"]):
        if record is not None:
            record.setdefault("h", []).append(x.copy())
        x, k, v = layer_full(x, layers[l], cfg, pos)
        if record is not None:
            record.setdefault("k", []).append(k)
            record.setdefault("v", []).append(v)
    return x


def cache_from_full_forward(record, m, n_layers_to_cache, cfg):
    """A 'fresh' cache for one request: the prefix rows of that request's own
    full forward (K/V and entering residuals) in the populate layout."""
    L = cfg["n_layers"]
    Lc = n_layers_to_cache
    n_h = min(Lc + 1, L)
    return {
        "k": np.stack([record["k"][l][:, :m] for l in range(Lc)]) if Lc else None,
        "v": np.stack([record["v"][l][:, :m] for l in range(Lc)]) if Lc else None,
        "h": np.stack([record["h"][l][:m] for l in range(n_h)]),
        "m": m,
    }
