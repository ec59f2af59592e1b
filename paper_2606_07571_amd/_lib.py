"""ctypes binding of libbicache.so: argument marshalling only.

Every step of the computation runs in the library's HIP kernels.  PyTorch
supplies device memory (weights, inputs, outputs, cache entries, workspace)
and the HIP stream (``torch.cuda.current_stream()``).  If the library is not
built, every call raises: there is no fallback path.
"""
import ctypes as C
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbicache.so")

STATUS = {0: "BC_OK", -1: "BC_E_INVALID", -2: "BC_E_NOT_FOUND", -3: "BC_E_OOM",
          -4: "BC_E_HIP", -5: "BC_E_STATE", -6: "BC_E_CAPACITY"}


class BiCacheError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("hidden", C.c_int), ("n_heads", C.c_int),
                ("n_kv_heads", C.c_int), ("head_dim", C.c_int), ("ffn", C.c_int),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float)]


class LayerWeights(C.Structure):
    _fields_ = [("w_qkv", C.c_void_p), ("w_o", C.c_void_p), ("w_gate_up", C.c_void_p),
                ("w_down", C.c_void_p), ("attn_norm", C.c_void_p), ("ffn_norm", C.c_void_p),
                ("b_qkv", C.c_void_p)]


_SIGS = {
    "bc_last_error": (C.c_char_p, []),
    "bc_model_create": (C.c_int, [C.POINTER(ModelConfig), C.POINTER(LayerWeights), C.c_int,
                                  C.POINTER(C.c_void_p)]),
    "bc_model_destroy": (C.c_int, [C.c_void_p]),
    "bc_prefix_cache_bytes": (C.c_size_t, [C.c_void_p, C.c_int, C.c_int]),
    "bc_cache_offset": (C.c_size_t, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                     C.c_int, C.c_int]),
    "bc_populate_workspace_bytes": (C.c_size_t, [C.c_void_p, C.c_int]),
    "bc_prefix_populate": (C.c_int, [C.c_void_p, C.c_uint64, C.c_void_p, C.c_int, C.c_int,
                                     C.c_void_p, C.c_size_t, C.c_void_p, C.c_size_t, C.c_void_p,
                                     C.POINTER(C.c_uint64), C.POINTER(C.c_int)]),
    "bc_prefix_lookup": (C.c_int, [C.c_void_p, C.c_uint64, C.POINTER(C.c_int), C.POINTER(C.c_int)]),
    "bc_prefix_invalidate": (C.c_int, [C.c_void_p, C.c_uint64]),
    "bc_cache_keys": (C.c_int, [C.c_void_p, C.POINTER(C.c_uint64), C.c_int, C.POINTER(C.c_int)]),
    "bc_prefix_key": (C.c_uint64, [C.POINTER(C.c_int32), C.c_size_t]),
    "bc_step_workspace_bytes": (C.c_size_t, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_int]),
    "bc_step_plan": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_int,
                               C.POINTER(C.c_int), C.POINTER(C.c_int), C.POINTER(C.c_int),
                               C.POINTER(C.c_int)]),
    "bc_step_forward": (C.c_int, [C.c_void_p, C.c_uint64, C.c_void_p, C.c_int, C.c_int, C.c_int,
                                  C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_shared_prefix_attention": (C.c_int, [C.c_void_p] * 6 + [C.c_int] * 6 + [C.c_float, C.c_void_p]),
    "bc_request_prefix_attention": (C.c_int, [C.c_void_p] * 6 + [C.c_int] * 6 + [C.c_float, C.c_void_p]),
    "bc_is_refresh_step": (C.c_int, [C.c_int, C.c_int]),
    "bc_profile_workspace_bytes": (C.c_size_t, [C.c_void_p, C.c_int, C.c_int, C.c_int]),
    "bc_profile_similarity": (C.c_int, [C.c_void_p, C.c_uint64, C.c_void_p, C.c_int, C.c_int, C.c_void_p,
                                        C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_cosine_workspace_bytes": (C.c_size_t, [C.c_long]),
    "bc_cosine_similarity": (C.c_int, [C.c_void_p, C.c_void_p, C.c_long, C.c_void_p, C.c_void_p,
                                       C.c_size_t, C.c_void_p]),
    "bc_cosine_similarity_noalloc": (C.c_int, [C.c_void_p, C.c_void_p, C.c_long, C.c_void_p, C.c_void_p]),
    "bc_shallow_depth": (C.c_int, [C.POINTER(C.c_double), C.c_int, C.c_double]),
    "bc_build_depth_table": (C.c_int, [C.POINTER(C.c_double), C.POINTER(C.c_int), C.c_int, C.c_int,
                                       C.POINTER(C.c_int)]),
    "bc_depth_lookup": (C.c_int, [C.POINTER(C.c_int), C.c_int, C.c_double]),
    "bc_step_multi_workspace_bytes": (C.c_size_t, [C.c_void_p, C.POINTER(C.c_uint64), C.POINTER(C.c_int),
                                                   C.c_int, C.c_int, C.c_int]),
    "bc_step_forward_multi": (C.c_int, [C.c_void_p, C.POINTER(C.c_uint64), C.POINTER(C.c_int), C.c_int,
                                        C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_size_t,
                                        C.c_void_p]),
    "bc_deep_store_reset": (C.c_int, [C.c_void_p, C.c_void_p]),
    "bc_deep_store_bytes": (C.c_size_t, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_int]),
    "bc_deep_store_offset": (C.c_size_t, [C.c_void_p] + [C.c_int] * 10),
    "bc_step_forward_deep": (C.c_int, [C.c_void_p, C.c_uint64, C.c_void_p, C.c_int, C.c_int, C.c_int,
                                       C.c_int, C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p,
                                       C.c_size_t, C.c_void_p]),
    "bc_profile_begin": (C.c_int, [C.c_void_p, C.c_uint]),
    "bc_profile_end": (C.c_int, [C.c_void_p, C.POINTER(C.c_double), C.POINTER(C.c_int)]),
}

# kernel classes of bc_profile_* (include/bicache.h)
KERNEL_CLASSES = ("rmsnorm", "qkv_rope", "attn_shared", "attn_full", "o_proj", "gate_up_swiglu",
                  "down", "other", "kv_similarity", "transition")

_lib = None


def lib():
    """The loaded library.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                               "(python -m paper_2606_07571_amd.build)")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status):
    if status != 0:
        raise BiCacheError(status, lib().bc_last_error().decode())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype, name):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return C.c_void_p(t.data_ptr())


def prefix_key(token_ids):
    """XXH64 (seed 0) of the token IDs as little-endian int32 (host only)."""
    import numpy as np
    a = np.ascontiguousarray(np.asarray(token_ids, dtype=np.int64).astype("<i4"))
    return int(lib().bc_prefix_key(a.ctypes.data_as(C.POINTER(C.c_int32)), a.size))


def shared_prefix_attention(q, k_pre, v_pre, k_suf, v_suf, scale=None, out=None):
    """One launch of the shared-prefix attention kernel.

    q [B,Hq,n_s,dh], k_pre/v_pre [Hkv,m,dh], k_suf/v_suf [B,Hkv,n_s,dh] (bf16,
    device); returns out fp32 [B,Hq,n_s,dh].
    """
    B, Hq, n_s, dh = q.shape
    Hkv, m = k_pre.shape[0], k_pre.shape[1]
    if scale is None:
        scale = dh ** -0.5
    if out is None:
        out = torch.empty((B, Hq, n_s, dh), dtype=torch.float32, device=q.device)
    bf = torch.bfloat16
    args = [_dev(q, bf, "q"), _dev(k_pre, bf, "k_pre"), _dev(v_pre, bf, "v_pre"),
            _dev(k_suf, bf, "k_suf"), _dev(v_suf, bf, "v_suf"), _dev(out, torch.float32, "out")]
    _check(lib().bc_shared_prefix_attention(*args, B, Hq, Hkv, m, n_s, dh, float(scale), _stream()))
    return out


def request_prefix_attention(q, k_pre, v_pre, k_suf, v_suf, scale=None, out=None):
    """One launch of the attention kernel with a per-request prefix.

    q [B,Hq,n_s,dh], k_pre/v_pre [B,Hkv,m,dh], k_suf/v_suf [B,Hkv,n_s,dh]
    (bf16, device); returns out fp32 [B,Hq,n_s,dh].
    """
    B, Hq, n_s, dh = q.shape
    Hkv, m = k_pre.shape[1], k_pre.shape[2]
    if scale is None:
        scale = dh ** -0.5
    if out is None:
        out = torch.empty((B, Hq, n_s, dh), dtype=torch.float32, device=q.device)
    bf = torch.bfloat16
    args = [_dev(q, bf, "q"), _dev(k_pre, bf, "k_pre"), _dev(v_pre, bf, "v_pre"),
            _dev(k_suf, bf, "k_suf"), _dev(v_suf, bf, "v_suf"), _dev(out, torch.float32, "out")]
    _check(lib().bc_request_prefix_attention(*args, B, Hq, Hkv, m, n_s, dh, float(scale), _stream()))
    return out


def is_refresh_step(t, delta):
    """Refresh schedule of Eq. 5 (host only): True when (t - 1) mod delta == 0."""
    r = lib().bc_is_refresh_step(t, delta)
    if r < 0:
        raise BiCacheError(-1, f"invalid step t={t} or refresh interval delta={delta}")
    return bool(r)


def cosine_similarity(a, b):
    """cos(a, b) of two bf16 device vectors (numel a multiple of 8), as a
    0-d fp64 device tensor."""
    n = a.numel()
    if b.numel() != n:
        raise ValueError("operands differ in size")
    wsb = int(lib().bc_cosine_workspace_bytes(n))
    if wsb == 0:
        raise BiCacheError(-1, f"n={n} must be a positive multiple of 8")
    ws = torch.empty(wsb, dtype=torch.uint8, device=a.device)
    out = torch.empty((), dtype=torch.float64, device=a.device)
    _check(lib().bc_cosine_similarity(_dev(a, torch.bfloat16, "a"), _dev(b, torch.bfloat16, "b"), n,
                                      C.c_void_p(out.data_ptr()), C.c_void_p(ws.data_ptr()), wsb, _stream()))
    return out


def cosine_similarity_noalloc(a, b, out):
    """cos(a, b) of two bf16 device vectors into ``out`` (a 0-d or 1-element
    fp64 device tensor) through the entry point that allocates nothing (its
    scratch is the library's static device array)."""
    n = a.numel()
    if b.numel() != n:
        raise ValueError("operands differ in size")
    _check(lib().bc_cosine_similarity_noalloc(_dev(a, torch.bfloat16, "a"), _dev(b, torch.bfloat16, "b"), n,
                                              _dev(out, torch.float64, "out"), _stream()))
    return out


def shallow_depth(sims, tau):
    """Sec. 4.2 rule on a host sequence of per-layer similarities (host only)."""
    arr = (C.c_double * max(len(sims), 1))(*[float(x) for x in sims])
    r = lib().bc_shallow_depth(arr, len(sims), float(tau))
    if r < 0:
        raise BiCacheError(-1, "invalid similarities")
    return r


def build_depth_table(ratios, depths, n_buckets=100):
    """Table T (host only): list of n_buckets + 1 ints, -1 where no data."""
    n = len(ratios)
    ra = (C.c_double * max(n, 1))(*[float(x) for x in ratios])
    da = (C.c_int * max(n, 1))(*[int(x) for x in depths])
    tab = (C.c_int * (n_buckets + 1))()
    _check(lib().bc_build_depth_table(ra, da, n, n_buckets, tab))
    return list(tab)


def depth_lookup(table, r):
    """d for shared-prefix ratio r from table T (host only)."""
    ta = (C.c_int * len(table))(*[int(x) for x in table])
    d = lib().bc_depth_lookup(ta, len(table) - 1, float(r))
    if d < 0:
        raise BiCacheError(-1, f"invalid lookup r={r}")
    return d


DEEP_MODES = {"refresh": 0, "reuse": 1}

_WEIGHT_KEYS = ("w_qkv", "w_o", "w_gate_up", "w_down", "attn_norm", "ffn_norm")


class Model:
    """A model over caller-owned device weights, with its prefix KV store.

    cfg: dict with n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn,
    rms_eps, rope_theta.  layers: list of dicts of bf16 device tensors
    (w_qkv, w_o, w_gate_up, w_down, attn_norm, ffn_norm).
    """

    def __init__(self, cfg, layers, cache_capacity=4):
        self.cfg = dict(cfg)
        self.layers = layers            # keep the weights alive
        c = ModelConfig(cfg["n_layers"], cfg["hidden"], cfg["n_heads"], cfg["n_kv_heads"],
                        cfg["head_dim"], cfg["ffn"], cfg["rms_eps"], cfg["rope_theta"])
        arr = (LayerWeights * len(layers))()
        for i, lw in enumerate(layers):
            for k in _WEIGHT_KEYS:
                setattr(arr[i], k, lw[k].data_ptr() if lw[k] is not None else None)
            bias = lw.get("b_qkv")
            arr[i].b_qkv = bias.data_ptr() if bias is not None else None
        h = C.c_void_p()
        _check(lib().bc_model_create(C.byref(c), arr, cache_capacity, C.byref(h)))
        self._h = h
        self._entries = {}              # key -> cache tensor (device memory of the entry)
        self._ws = None

    def close(self):
        if self._h:
            lib().bc_model_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- cache
    def cache_bytes(self, m, n_layers_to_cache):
        return int(lib().bc_prefix_cache_bytes(self._h, m, n_layers_to_cache))

    def cache_offset(self, m, n_layers_to_cache, layer, part, head, pos, dim):
        return int(lib().bc_cache_offset(self._h, m, n_layers_to_cache, layer, part, head, pos, dim))

    def _workspace(self, nbytes, device):
        if self._ws is None or self._ws.numel() < nbytes or self._ws.device != device:
            self._ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        return self._ws

    def populate(self, key, x_prefix, n_layers_to_cache=None):
        """Prefix-only forward of x_prefix [m, h] (bf16, device) into a new cache
        entry under ``key``.  Returns the evicted key or None."""
        L = self.cfg["n_layers"]
        Lc = L if n_layers_to_cache is None else n_layers_to_cache
        m = x_prefix.shape[0]
        nbytes = self.cache_bytes(m, Lc)
        if nbytes == 0:
            raise BiCacheError(-1, f"invalid prefix shape m={m} Lc={Lc}")
        mem = torch.empty(nbytes, dtype=torch.uint8, device=x_prefix.device)
        wsb = int(lib().bc_populate_workspace_bytes(self._h, m))
        ws = self._workspace(wsb, x_prefix.device)
        ek, ev = C.c_uint64(0), C.c_int(0)
        _check(lib().bc_prefix_populate(self._h, C.c_uint64(key), _dev(x_prefix, torch.bfloat16, "x_prefix"),
                                        m, Lc, C.c_void_p(mem.data_ptr()), nbytes,
                                        C.c_void_p(ws.data_ptr()), ws.numel(), _stream(),
                                        C.byref(ek), C.byref(ev)))
        self._entries[key] = mem
        if ev.value:
            self._entries.pop(ek.value, None)
            return ek.value
        return None

    def lookup(self, key):
        m, n = C.c_int(), C.c_int()
        st = lib().bc_prefix_lookup(self._h, C.c_uint64(key), C.byref(m), C.byref(n))
        if st == -2:
            return None
        _check(st)
        return m.value, n.value

    def invalidate(self, key):
        _check(lib().bc_prefix_invalidate(self._h, C.c_uint64(key)))
        self._entries.pop(key, None)

    def cache_keys(self):
        n = C.c_int()
        _check(lib().bc_cache_keys(self._h, None, 0, C.byref(n)))
        buf = (C.c_uint64 * max(n.value, 1))()
        _check(lib().bc_cache_keys(self._h, buf, n.value, C.byref(n)))
        return [int(buf[i]) for i in range(n.value)]

    def cache_tensor(self, key):
        return self._entries[key]

    # ---------------------------------------------------------------- profiling
    def profile_begin(self, classes=KERNEL_CLASSES):
        """Time every later launch of the named kernel classes with HIP events."""
        mask = 0
        for c in classes:
            mask |= 1 << KERNEL_CLASSES.index(c)
        _check(lib().bc_profile_begin(self._h, mask))

    def profile_end(self):
        """Returns {class: (total_ms, launches)} of the timed launches."""
        n = len(KERNEL_CLASSES)
        ms, cnt = (C.c_double * n)(), (C.c_int * n)()
        _check(lib().bc_profile_end(self._h, ms, cnt))
        return {KERNEL_CLASSES[i]: (ms[i], cnt[i]) for i in range(n) if cnt[i]}

    # ---------------------------------------------------------------- step
    def step_workspace_bytes(self, m, B, n_s, d):
        return int(lib().bc_step_workspace_bytes(self._h, m, B, n_s, d))

    def step_plan(self, m, B, n_s, d):
        L = self.cfg["n_layers"]
        rows, pos, kv = (C.c_int * L)(), (C.c_int * L)(), (C.c_int * L)()
        rh = C.c_int()
        _check(lib().bc_step_plan(self._h, m, B, n_s, d, rows, pos, kv, C.byref(rh)))
        return list(rows), list(pos), list(kv), rh.value

    def step_multi(self, keys, counts, x_suffix, d, out=None):
        """Step of a batch over several cached prefixes: group g is counts[g]
        consecutive requests of x_suffix [B, n_s, h] (bf16, device) sharing the
        prefix keys[g].  Returns the fp32 suffix rows [B, n_s, h]."""
        B, n_s, h = x_suffix.shape
        G = len(keys)
        if len(counts) != G or sum(counts) != B:
            raise ValueError(f"counts {list(counts)} do not cover the batch of {B}")
        karr = (C.c_uint64 * G)(*[int(k) for k in keys])
        carr = (C.c_int * G)(*[int(c) for c in counts])
        wsb = int(lib().bc_step_multi_workspace_bytes(self._h, karr, carr, G, n_s, d))
        if wsb == 0:
            missing = [k for k in keys if self.lookup(k) is None]
            if missing:
                raise BiCacheError(-2, f"keys {[hex(k) for k in missing]} are not cached")
            raise BiCacheError(-1, f"invalid multi-prefix step counts={list(counts)} n_s={n_s} d={d}")
        ws = self._workspace(wsb, x_suffix.device)
        if out is None:
            out = torch.empty((B, n_s, h), dtype=torch.float32, device=x_suffix.device)
        _check(lib().bc_step_forward_multi(self._h, karr, carr, G, _dev(x_suffix, torch.bfloat16, "x_suffix"),
                                           n_s, d, _dev(out, torch.float32, "out"),
                                           C.c_void_p(ws.data_ptr()), ws.numel(), _stream()))
        return out

    def profile_similarity(self, key, x_suffix, sims=None):
        """sim_{l,1} (Eq. 3) of every request of x_suffix [B, n_s, h] (bf16,
        device) and every layer, over the cached prefix ``key`` (all L layers
        cached).  Returns a device fp64 tensor [B, L]."""
        B, n_s, h = x_suffix.shape
        got = self.lookup(key)
        if got is None:
            raise BiCacheError(-2, f"key {key:#x} is not cached")
        wsb = int(lib().bc_profile_workspace_bytes(self._h, got[0], B, n_s))
        if wsb == 0:
            raise BiCacheError(-1, f"invalid profiling shape B={B} n_s={n_s}")
        ws = self._workspace(wsb, x_suffix.device)
        if sims is None:
            sims = torch.empty((B, self.cfg["n_layers"]), dtype=torch.float64, device=x_suffix.device)
        _check(lib().bc_profile_similarity(self._h, C.c_uint64(key), _dev(x_suffix, torch.bfloat16, "x_suffix"),
                                           B, n_s, _dev(sims, torch.float64, "sims"),
                                           C.c_void_p(ws.data_ptr()), ws.numel(), _stream()))
        return sims

    def deep_store_bytes(self, m, B, n_s, d):
        return int(lib().bc_deep_store_bytes(self._h, m, B, n_s, d))

    def deep_store_offset(self, m, B, n_s, d, layer, part, req, head, pos, dim):
        return int(lib().bc_deep_store_offset(self._h, m, B, n_s, d, layer, part, req, head, pos, dim))

    def new_deep_store(self, key, B, n_s, d, device="cuda"):
        """Device memory for the deep store of a batch (None when d = L)."""
        got = self.lookup(key)
        if got is None:
            raise BiCacheError(-2, f"key {key:#x} is not cached")
        nbytes = self.deep_store_bytes(got[0], B, n_s, d)
        if nbytes == 0:
            return None
        store = torch.empty(nbytes, dtype=torch.uint8, device=device)
        # the allocator may hand out the address of an earlier, tagged store
        _check(lib().bc_deep_store_reset(self._h, C.c_void_p(store.data_ptr())))
        return store

    def step(self, key, x_suffix, d, out=None, deep=None, deep_store=None):
        """Step forward of x_suffix [B, n_s, h] (bf16, device) at reuse depth d.

        deep=None runs bc_step_forward; deep="refresh" / "reuse" runs
        bc_step_forward_deep in that mode with ``deep_store`` (a uint8 device
        tensor from new_deep_store, or None).  Returns the fp32 suffix rows of
        the final residual [B, n_s, h]."""
        B, n_s, h = x_suffix.shape
        got = self.lookup(key)
        if got is None:
            raise BiCacheError(-2, f"key {key:#x} is not cached")
        m = got[0]
        wsb = self.step_workspace_bytes(m, B, n_s, d)
        if wsb == 0:
            raise BiCacheError(-1, f"invalid step shape B={B} n_s={n_s} d={d}")
        ws = self._workspace(wsb, x_suffix.device)
        if out is None:
            out = torch.empty((B, n_s, h), dtype=torch.float32, device=x_suffix.device)
        xs = _dev(x_suffix, torch.bfloat16, "x_suffix")
        o = _dev(out, torch.float32, "out")
        wsp = C.c_void_p(ws.data_ptr())
        if deep is None:
            _check(lib().bc_step_forward(self._h, C.c_uint64(key), xs, B, n_s, d, o, wsp, ws.numel(),
                                         _stream()))
            return out
        if deep not in DEEP_MODES:
            raise ValueError(f"deep must be one of {sorted(DEEP_MODES)}, got {deep!r}")
        if deep_store is None:
            sp, sb = None, 0
        else:
            sp, sb = _dev(deep_store, torch.uint8, "deep_store"), deep_store.numel()
        _check(lib().bc_step_forward_deep(self._h, C.c_uint64(key), xs, B, n_s, d, DEEP_MODES[deep],
                                          sp, sb, o, wsp, ws.numel(), _stream()))
        return out
