"""Host-side checks of the C ABI (no GPU): exports, argument validation, key
hash, cache layout offsets, step work accounting, FIFO bookkeeping."""
import ctypes as C
import os
import re

import numpy as np
import pytest
import xxhash

from oracle.cache_table import FifoTable
from oracle.xxh64 import prefix_key as oracle_prefix_key

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bicache.h")

pytest.importorskip("torch")
import paper_2606_07571_amd as bc  # noqa: E402
from paper_2606_07571_amd import _lib  # noqa: E402


def _declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bc_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = bc.lib()
    syms = _declared_symbols()
    assert len(syms) >= 15
    for s in syms:
        assert hasattr(L, s), f"{s} not exported"


def test_kernel_classes_match_header_enum():
    # the binding names the timing classes of bc_profile_begin/end in enum order
    text = open(HEADER).read()
    enum = dict((k, int(v)) for k, v in re.findall(r"\b(BC_K_[A-Z_]+)\s*=\s*(\d+)", text))
    assert enum.pop("BC_K_COUNT") == len(_lib.KERNEL_CLASSES)
    assert sorted(enum.values()) == list(range(len(_lib.KERNEL_CLASSES)))
    assert _lib.KERNEL_CLASSES[enum["BC_K_TRANSITION"]] == "transition"
    assert _lib.KERNEL_CLASSES[enum["BC_K_KVSIM"]] == "kv_similarity"
    assert _lib.KERNEL_CLASSES[enum["BC_K_RMSNORM"]] == "rmsnorm"


def test_prefix_key_matches_xxhash_and_oracle():
    rng = np.random.default_rng(0)
    for n in (0, 1, 7, 8, 9, 31, 32, 33, 1536, 8192):
        ids = rng.integers(-2**31, 2**31 - 1, size=n)
        k = bc.prefix_key(ids)
        assert k == xxhash.xxh64_intdigest(ids.astype("<i4").tobytes(), seed=0)
        if n <= 64:
            assert k == oracle_prefix_key(ids)


CFG = dict(n_layers=3, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
           rms_eps=1e-5, rope_theta=500000.0)
FAKE = 1 << 20      # a non-null fake device address: never dereferenced by these calls


def _fake_layers(n):
    return [{k: None for k in _lib._WEIGHT_KEYS} for _ in range(n)]


def _model(cfg=CFG, cap=4):
    arr = (_lib.LayerWeights * cfg["n_layers"])()
    for i in range(cfg["n_layers"]):
        for k in _lib._WEIGHT_KEYS:
            setattr(arr[i], k, FAKE)
    c = _lib.ModelConfig(*[cfg[k] for k in ("n_layers", "hidden", "n_heads", "n_kv_heads",
                                             "head_dim", "ffn", "rms_eps", "rope_theta")])
    h = C.c_void_p()
    st = bc.lib().bc_model_create(C.byref(c), arr, cap, C.byref(h))
    return st, h


def test_model_create_validation():
    st, h = _model()
    assert st == 0
    assert bc.lib().bc_model_destroy(h) == 0
    for bad in (dict(n_layers=0), dict(hidden=100), dict(head_dim=96), dict(n_kv_heads=3),
                dict(ffn=100), dict(hidden=16384)):
        st, _ = _model(dict(CFG, **bad))
        assert st == -1, bad
        assert "invalid model config" in bc.lib().bc_last_error().decode()
    st, _ = _model(cap=0)
    assert st == -1
    # a null weight pointer
    arr = (_lib.LayerWeights * 3)()
    c = _lib.ModelConfig(3, 256, 4, 2, 64, 512, 1e-5, 5e5)
    h = C.c_void_p()
    assert bc.lib().bc_model_create(C.byref(c), arr, 2, C.byref(h)) == -1


def test_cache_layout_offsets():
    st, h = _model()
    L = bc.lib()
    m, Lc = 129, 2
    Hkv, dh, hid = 2, 64, 256
    kv_layer = Hkv * m * dh * 2
    h_off = -(-(Lc * 2 * kv_layer) // 256) * 256
    n_h = min(Lc + 1, 3)
    assert L.bc_prefix_cache_bytes(h, m, Lc) == h_off + n_h * m * hid * 4
    for (layer, part, head, pos, dim) in [(0, 0, 0, 0, 0), (1, 1, 1, 128, 63), (0, 1, 1, 5, 7)]:
        exp = (layer * 2 + part) * kv_layer + ((head * m + pos) * dh + dim) * 2
        assert L.bc_cache_offset(h, m, Lc, layer, part, head, pos, dim) == exp
    for (layer, pos, dim) in [(0, 0, 0), (2, 128, 255), (1, 3, 4)]:
        exp = h_off + layer * m * hid * 4 + (pos * hid + dim) * 4
        assert L.bc_cache_offset(h, m, Lc, layer, 2, 0, pos, dim) == exp
    bad = (1 << 64) - 1
    assert L.bc_cache_offset(h, m, Lc, 2, 0, 0, 0, 0) == bad      # layer >= Lc
    assert L.bc_cache_offset(h, m, Lc, 3, 2, 0, 0, 0) == bad      # H$ index > min(Lc, L-1)
    assert L.bc_cache_offset(h, m, Lc, 0, 0, 2, 0, 0) == bad      # head >= Hkv
    assert L.bc_cache_offset(h, m, Lc, 0, 0, 0, m, 0) == bad      # pos >= m
    assert L.bc_cache_offset(h, m, Lc, 0, 3, 0, 0, 0) == bad      # no such part
    assert L.bc_prefix_cache_bytes(h, 0, 1) == 0 and L.bc_prefix_cache_bytes(h, 4, 4) == 0
    L.bc_model_destroy(h)


def test_step_plan_accounting():
    st, h = _model()
    L = bc.lib()
    m, B, n_s = 129, 3, 65
    for d in range(4):
        rows, pos, kv = (C.c_int * 3)(), (C.c_int * 3)(), (C.c_int * 3)()
        rh = C.c_int()
        assert L.bc_step_plan(h, m, B, n_s, d, rows, pos, kv, C.byref(rh)) == 0
        assert list(rows) == [B * n_s if l < d else B * (m + n_s) for l in range(3)]
        assert list(pos) == [m if l < d else 0 for l in range(3)]
        assert list(kv) == [1 if l < d else 0 for l in range(3)]
        assert rh.value == (d if d < 3 else -1)
    assert L.bc_step_plan(h, m, B, n_s, 4, None, None, None, None) == -1
    assert L.bc_step_plan(h, m, B, n_s, -1, None, None, None, None) == -1
    assert L.bc_step_plan(h, m, 0, n_s, 1, None, None, None, None) == -1
    # the workspace grows with the deep part
    assert L.bc_step_workspace_bytes(h, m, B, n_s, 3) < L.bc_step_workspace_bytes(h, m, B, n_s, 0)
    assert L.bc_step_workspace_bytes(h, m, B, n_s, 5) == 0
    L.bc_model_destroy(h)


def test_entry_point_validation_without_device_work():
    st, h = _model(cap=2)
    L = bc.lib()
    ev, evk = C.c_int(7), C.c_uint64(7)
    big = 1 << 40
    # m = 0, Lc > L, short cache, misaligned cache, short workspace, null input
    assert L.bc_prefix_populate(h, 1, FAKE, 0, 1, FAKE, big, FAKE, big, None, C.byref(evk), C.byref(ev)) == -1
    assert ev.value == 0 and evk.value == 0
    assert L.bc_prefix_populate(h, 1, FAKE, 8, 4, FAKE, big, FAKE, big, None, None, None) == -1
    assert L.bc_prefix_populate(h, 1, FAKE, 8, 3, FAKE, 16, FAKE, big, None, None, None) == -1
    assert L.bc_prefix_populate(h, 1, FAKE, 8, 3, FAKE + 8, big, FAKE, big, None, None, None) == -1
    assert L.bc_prefix_populate(h, 1, FAKE, 8, 3, FAKE, big, FAKE, 16, None, None, None) == -1
    assert L.bc_prefix_populate(h, 1, None, 8, 3, FAKE, big, FAKE, big, None, None, None) == -1
    # nothing was inserted
    n = C.c_int()
    assert L.bc_cache_keys(h, None, 0, C.byref(n)) == 0 and n.value == 0
    # miss paths
    assert L.bc_step_forward(h, 1, FAKE, 2, 4, 1, FAKE, FAKE, big, None) == -2
    assert "not cached" in L.bc_last_error().decode()
    assert L.bc_prefix_lookup(h, 1, None, None) == -2
    assert L.bc_prefix_invalidate(h, 1) == -2
    # attention-only entry point
    A = L.bc_shared_prefix_attention
    assert A(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 4, 4, 8, 4, 96, 0.1, None) == -1   # dh
    assert A(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 6, 4, 8, 4, 64, 0.1, None) == -1   # Hq % Hkv
    assert A(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 4, 4, 8, 4, 64, 0.1, None) == -1   # B
    assert A(FAKE, None, FAKE, FAKE, FAKE, FAKE, 2, 4, 4, 8, 4, 64, 0.1, None) == -1   # null prefix, m > 0
    L.bc_model_destroy(h)


def test_refresh_schedule_matches_oracle():
    from oracle.transformer import is_refresh_step
    for delta in (1, 2, 3, 16, 64):
        for t in range(1, 200):
            assert bc.is_refresh_step(t, delta) == is_refresh_step(t, delta)
    L = bc.lib()
    assert L.bc_is_refresh_step(0, 16) == -1 and L.bc_is_refresh_step(1, 0) == -1
    assert L.bc_is_refresh_step(-5, 3) == -1
    with pytest.raises(bc.BiCacheError):
        bc.is_refresh_step(0, 16)


def test_deep_store_layout_offsets():
    st, h = _model()
    L = bc.lib()
    m, B, n_s = 129, 3, 65
    Hkv, dh, nl = 2, 64, 3
    N = m + n_s
    for d in range(nl + 1):
        part = B * Hkv * N * dh * 2
        # the K/V blocks, then a 256-byte header (the refresh's tag) when there are deep layers
        assert L.bc_deep_store_bytes(h, m, B, n_s, d) == ((nl - d) * 2 * part + 256 if d < nl else 0)
        assert part % 256 == 0
        for (layer, pt, req, head, pos, dim) in [(d, 0, 0, 0, 0, 0), (nl - 1, 1, B - 1, Hkv - 1, N - 1, dh - 1),
                                                 (d, 1, 1, 0, m, 3)]:
            off = L.bc_deep_store_offset(h, m, B, n_s, d, layer, pt, req, head, pos, dim)
            if d == nl:
                assert off == (1 << 64) - 1
                continue
            exp = (2 * (layer - d) + pt) * part + (((req * Hkv + head) * N + pos) * dh + dim) * 2
            assert off == exp
    bad = (1 << 64) - 1
    d = 1
    assert L.bc_deep_store_offset(h, m, B, n_s, d, 0, 0, 0, 0, 0, 0) == bad      # shallow layer
    assert L.bc_deep_store_offset(h, m, B, n_s, d, 3, 0, 0, 0, 0, 0) == bad      # layer >= L
    assert L.bc_deep_store_offset(h, m, B, n_s, d, 1, 2, 0, 0, 0, 0) == bad      # no such part
    assert L.bc_deep_store_offset(h, m, B, n_s, d, 1, 0, B, 0, 0, 0) == bad      # req >= B
    assert L.bc_deep_store_offset(h, m, B, n_s, d, 1, 0, 0, 0, N, 0) == bad      # pos >= N
    assert L.bc_deep_store_bytes(h, m, B, n_s, 4) == 0
    assert L.bc_deep_store_bytes(h, 0, B, n_s, 1) == 0
    # the last element ends the K/V blocks; the 256-byte header follows
    last = L.bc_deep_store_offset(h, m, B, n_s, 0, nl - 1, 1, B - 1, Hkv - 1, N - 1, dh - 1)
    assert last + 2 + 256 == L.bc_deep_store_bytes(h, m, B, n_s, 0)
    L.bc_model_destroy(h)


def test_deep_step_validation_without_device_work():
    st, h = _model()
    L = bc.lib()
    big = 1 << 40
    S = L.bc_step_forward_deep
    # miss first, then mode checks never reach the device
    assert S(h, 1, FAKE, 2, 4, 1, 1, FAKE, big, FAKE, FAKE, big, None) == -2
    assert S(h, 1, FAKE, 2, 4, 1, 7, FAKE, big, FAKE, FAKE, big, None) == -1
    assert "deep mode" in L.bc_last_error().decode()
    assert S(h, 1, None, 2, 4, 1, 0, FAKE, big, FAKE, FAKE, big, None) == -1
    assert L.bc_deep_store_reset(h, FAKE) == 0 and L.bc_deep_store_reset(None, FAKE) == -1
    A = L.bc_request_prefix_attention
    assert A(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 4, 4, 8, 4, 96, 0.1, None) == -1   # dh
    assert A(FAKE, None, FAKE, FAKE, FAKE, FAKE, 2, 4, 4, 8, 4, 64, 0.1, None) == -1   # null prefix, m > 0
    L.bc_model_destroy(h)


def test_depth_rule_and_table_match_oracle():
    from oracle import profiling as P
    rng = np.random.default_rng(5)
    for _ in range(200):
        L = int(rng.integers(0, 40))
        sims = list(1 - np.abs(rng.normal(scale=0.03, size=L)))
        tau = float(rng.choice([0.9, 0.95, 0.97, 0.99]))
        assert bc.shallow_depth(sims, tau) == P.shallow_depth(sims, tau)
    n_buckets = 100
    ks = rng.integers(1, n_buckets + 1, size=500)
    ks[ks == 37] = 38                       # leave bucket 37 without data
    ratios = [k / n_buckets for k in ks]
    depths = [int(x) for x in rng.integers(0, 33, size=500)]
    T = bc.build_depth_table(ratios, depths, n_buckets)
    assert T == P.build_table(ratios, depths, n_buckets)
    assert T[37] == -1
    for r in list(np.linspace(0, 1, 401)) + [0.37, 0.3699999, 0.75, 1.0]:
        assert bc.depth_lookup(T, r) == P.lookup_depth(T, r), r
    with pytest.raises(bc.BiCacheError):
        bc.build_depth_table([0.333], [1], 100)
    with pytest.raises(bc.BiCacheError):
        bc.build_depth_table([0.5], [-1], 100)
    L = bc.lib()
    assert L.bc_cosine_workspace_bytes(12) == 0 and L.bc_cosine_workspace_bytes(0) == 0
    assert L.bc_cosine_workspace_bytes(8 * 8192) > 0


# ------------------------------------------------------------ FIFO bookkeeping

@pytest.fixture(scope="module")
def host_table():
    path = os.path.join(ROOT, "tests", "native", "libbicache_table_host.so")
    if not os.path.exists(path):
        pytest.skip("host table library not built")
    T = C.CDLL(path)
    T.bct_create.restype = C.c_void_p
    T.bct_create.argtypes = [C.c_int]
    T.bct_destroy.argtypes = [C.c_void_p]
    T.bct_insert.argtypes = [C.c_void_p, C.c_uint64, C.c_int, C.POINTER(C.c_uint64)]
    T.bct_erase.argtypes = [C.c_void_p, C.c_uint64]
    T.bct_lookup.argtypes = [C.c_void_p, C.c_uint64]
    T.bct_keys.argtypes = [C.c_void_p, C.POINTER(C.c_uint64), C.c_int]
    T.bct_xxh64.restype = C.c_uint64
    T.bct_xxh64.argtypes = [C.c_void_p, C.c_uint64, C.c_uint64]
    return T


@pytest.mark.parametrize("cap", [1, 2, 5])
def test_fifo_table_matches_model(host_table, cap):
    T = host_table
    t = T.bct_create(cap)
    ref = FifoTable(cap)
    rng = np.random.default_rng(cap)
    keys = [int(x) for x in rng.integers(0, 2**64 - 1, size=12, dtype=np.uint64)]
    for step in range(400):
        k = keys[rng.integers(len(keys))]
        op = rng.integers(3)
        if op == 0:
            ev = C.c_uint64()
            r = T.bct_insert(t, k, step, C.byref(ev))
            try:
                e = ref.insert(k, step)
                assert r == (1 if e is not None else 0)
                if e is not None:
                    assert ev.value == e
            except KeyError:
                assert r == -1
        elif op == 1:
            assert T.bct_erase(t, k) == (1 if ref.invalidate(k) else 0)
        else:
            meta = ref.lookup(k)
            assert T.bct_lookup(t, k) == (-1 if meta is None else meta)
        buf = (C.c_uint64 * 16)()
        n = T.bct_keys(t, buf, 16)
        assert [buf[i] for i in range(n)] == ref.order()
    T.bct_destroy(t)


def test_native_xxh64_matches_library(host_table):
    rng = np.random.default_rng(9)
    for n in list(range(0, 80)) + [1000]:
        data = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        for seed in (0, 12345):
            assert host_table.bct_xxh64(data, n, seed) == xxhash.xxh64_intdigest(data, seed=seed)


def test_misaligned_device_pointers_are_refused():
    """Every device pointer must be 16-byte aligned (the kernels move 16-byte
    vectors); a pointer 8 bytes off is refused before anything is enqueued."""
    L = bc.lib()
    MIS = FAKE + 8
    # weights at model creation, each of the seven pointers in turn
    for k in list(_lib._WEIGHT_KEYS) + ["b_qkv"]:
        arr = (_lib.LayerWeights * CFG["n_layers"])()
        for i in range(CFG["n_layers"]):
            for kk in _lib._WEIGHT_KEYS:
                setattr(arr[i], kk, FAKE)
        setattr(arr[1], k, MIS)
        c = _lib.ModelConfig(*[CFG[x] for x in ("n_layers", "hidden", "n_heads", "n_kv_heads",
                                                 "head_dim", "ffn", "rms_eps", "rope_theta")])
        h = C.c_void_p()
        assert L.bc_model_create(C.byref(c), arr, 2, C.byref(h)) == -1, k
        assert "16-byte aligned" in L.bc_last_error().decode()
    st, h = _model()
    big = 1 << 40
    assert L.bc_prefix_populate(h, 1, MIS, 8, 3, FAKE, big, FAKE, big, None, None, None) == -1
    assert "16-byte" in L.bc_last_error().decode()
    # step inputs and outputs (refused before the key is even looked up)
    assert L.bc_step_forward(h, 1, MIS, 2, 4, 1, FAKE, FAKE, big, None) == -1
    assert L.bc_step_forward(h, 1, FAKE, 2, 4, 1, MIS, FAKE, big, None) == -1
    S = L.bc_step_forward_deep
    assert S(h, 1, MIS, 2, 4, 1, 0, FAKE, big, FAKE, FAKE, big, None) == -1
    assert S(h, 1, FAKE, 2, 4, 1, 1, FAKE, big, MIS, FAKE, big, None) == -1
    keys, counts = (C.c_uint64 * 1)(1), (C.c_int * 1)(2)
    assert L.bc_step_forward_multi(h, keys, counts, 1, MIS, 4, 1, FAKE, FAKE, big, None) == -1
    assert L.bc_profile_similarity(h, 1, MIS, 2, 4, FAKE, FAKE, big, None) == -1
    assert L.bc_profile_similarity(h, 1, FAKE, 2, 4, MIS, FAKE, big, None) == -1
    # attention operands, each in turn
    for A in (L.bc_shared_prefix_attention, L.bc_request_prefix_attention):
        for i in range(6):
            ptrs = [FAKE] * 6
            ptrs[i] = MIS
            assert A(*ptrs, 2, 4, 4, 8, 4, 64, 0.1, None) == -1, i
            assert "16-byte" in L.bc_last_error().decode()
    # the cosine reduction
    ws = L.bc_cosine_workspace_bytes(64)
    assert L.bc_cosine_similarity(MIS, FAKE, 64, FAKE, FAKE, ws, None) == -1
    assert L.bc_cosine_similarity(FAKE, FAKE, 64, MIS, FAKE, ws, None) == -1
    L.bc_model_destroy(h)


def test_destroyed_handle_is_refused():
    """A handle used after bc_model_destroy is refused, never dereferenced."""
    L = bc.lib()
    st, h = _model()
    assert st == 0
    assert L.bc_model_destroy(h) == 0
    assert L.bc_model_destroy(h) == -1
    assert "destroyed" in L.bc_last_error().decode()
    assert L.bc_prefix_lookup(h, 1, None, None) == -1
    assert L.bc_prefix_invalidate(h, 1) == -1
    n = C.c_int()
    assert L.bc_cache_keys(h, None, 0, C.byref(n)) == -1
    assert L.bc_step_forward(h, 1, FAKE, 2, 4, 1, FAKE, FAKE, 1 << 40, None) == -1
    assert L.bc_step_workspace_bytes(h, 8, 2, 4, 1) == 0
    assert L.bc_prefix_cache_bytes(h, 8, 1) == 0
    assert L.bc_deep_store_bytes(h, 8, 2, 4, 1) == 0
    assert L.bc_profile_begin(h, 1) == -1
    assert L.bc_deep_store_reset(h, FAKE) == -1
    # an unknown (never created) handle as well
    bogus = C.c_void_p(FAKE)
    assert L.bc_prefix_lookup(bogus, 1, None, None) == -1
    assert L.bc_model_destroy(bogus) == -1


def test_failed_host_allocation_leaves_table_unchanged(host_table):
    """An allocation failure inside an insert (std::bad_alloc, which the
    library reports as BC_E_OOM) evicts nothing and changes nothing."""
    T = host_table
    T.bct_fail_allocs_after.argtypes = [C.c_long]
    t = T.bct_create(2)
    ev = C.c_uint64()
    assert T.bct_insert(t, 11, 1, C.byref(ev)) == 0
    assert T.bct_insert(t, 22, 2, C.byref(ev)) == 0
    buf = (C.c_uint64 * 4)()
    T.bct_fail_allocs_after(0)
    try:
        r = T.bct_insert(t, 33, 3, C.byref(ev))
    finally:
        T.bct_fail_allocs_after(-1)
    assert r == -2
    n = T.bct_keys(t, buf, 4)
    assert [buf[i] for i in range(n)] == [11, 22]     # nothing evicted
    assert T.bct_lookup(t, 33) == -1 and T.bct_lookup(t, 11) == 1
    assert T.bct_insert(t, 33, 3, C.byref(ev)) == 1 and ev.value == 11
    n = T.bct_keys(t, buf, 4)
    assert [buf[i] for i in range(n)] == [22, 33]
    T.bct_destroy(t)


def test_noalloc_cosine_validation_without_device_work():
    """The allocation-free cosine refuses, before any device work, sizes beyond
    its static scratch (130,146,304 elements), bad sizes and misaligned or
    null pointers."""
    L = bc.lib()
    N = L.bc_cosine_similarity_noalloc
    assert N(FAKE, FAKE, 130_146_304 + 8, FAKE, None) == -6
    assert "static scratch" in L.bc_last_error().decode()
    assert N(FAKE, FAKE, 12, FAKE, None) == -1
    assert N(FAKE, FAKE, 0, FAKE, None) == -1
    assert N(FAKE + 8, FAKE, 64, FAKE, None) == -1
    assert N(FAKE, FAKE, 64, FAKE + 8, None) == -1
    assert N(None, FAKE, 64, FAKE, None) == -1
