/*
 * bicache.h -- C ABI of libbicache.so: BiCache's shared-prefix denoising step
 * for diffusion language models on AMD Instinct MI355X (gfx950).
 *
 * The method (BiCache, "bidirectional prefix caching"):
 *   - A shared prefix p is run once on its own ("populate", Sec. 5.2: on a
 *     miss the KVs of p are computed at the first step for all layers and
 *     stored in the KV store H under the key h(p)).
 *   - A denoising step of a batch of requests that share p runs the layers
 *     shallower than the reuse depth d on the suffix rows only, attending over
 *     the cached prefix K/V plus the request's own suffix K/V (Eq. 4), and
 *     recomputes the prefix in the layers at or beyond d with full
 *     bidirectional attention (refresh case of Eq. 5).  The paper's depth b
 *     (1-based, layers l <= b reuse the cache) is d here (0-based, l < d).
 *
 * Conventions for every entry point:
 *   - Device buffers are allocated and owned by the caller.  The library never
 *     allocates or frees device memory; it keeps host-side metadata only (its
 *     one device array is the static scratch of bc_cosine_similarity_noalloc).
 *   - Tensors are dense, row-major, bf16 = IEEE bfloat16 bits (uint16), fp32 =
 *     IEEE binary32.  Every device pointer must be 16-byte aligned (the kernels
 *     move 16-byte vectors); a misaligned one returns BC_E_INVALID.
 *   - `stream` is a hipStream_t passed as an opaque pointer (NULL = the null
 *     stream).  Every device operation is enqueued asynchronously on it; no
 *     call synchronizes the host.
 *   - No C++ exception crosses this boundary.  Every call returns a bc_status;
 *     bc_last_error() gives a message for the calling thread's last failure.
 *     A failed host allocation returns BC_E_OOM; a model handle that was
 *     destroyed (or never created) returns BC_E_INVALID.
 *     All arguments are validated before anything is enqueued, so a call that
 *     returns BC_E_INVALID / BC_E_NOT_FOUND / BC_E_STATE has no side effect.
 *   - A bc_model is not thread-safe: calls on one model must not overlap.
 *
 * The layer is a pre-norm transformer block: RMSNorm, fused Q/K/V projection
 * (Eq. 1, optionally with a bias), rotate-half RoPE, unmasked attention
 * (Eq. 2), output projection plus residual, RMSNorm, SwiGLU FFN plus
 * residual; no other biases.  The residual
 * stream is fp32; GEMM and attention operands are bf16 with fp32
 * accumulation.
 */
#ifndef BICACHE_H
#define BICACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BC_OK = 0,
  BC_E_INVALID = -1,   /* bad argument: null pointer, size, range or shape */
  BC_E_NOT_FOUND = -2, /* step/lookup on a key that is not cached (the paper's miss) */
  BC_E_OOM = -3,       /* host allocation failed */
  BC_E_HIP = -4,       /* a HIP runtime call failed (includes earlier async faults) */
  BC_E_STATE = -5,     /* operation not allowed in this state (e.g. key already cached) */
  BC_E_CAPACITY = -6   /* a size is beyond what a kernel supports */
} bc_status;

/* Message of the calling thread's last failed call ("" if none).  The pointer
 * stays valid until the next call on the same thread. */
const char* bc_last_error(void);

/* ------------------------------------------------------------------ model */

typedef struct {
  int n_layers;    /* L >= 1 */
  int hidden;      /* h, multiple of 64 */
  int n_heads;     /* Hq query heads */
  int n_kv_heads;  /* Hkv KV heads, Hq % Hkv == 0 (grouped-query attention:
                      query head j reads KV head j / (Hq/Hkv)) */
  int head_dim;    /* dh: 64 or 128 */
  int ffn;         /* F, SwiGLU width, multiple of 64 */
  float rms_eps;   /* RMSNorm epsilon */
  float rope_theta;/* RoPE base; pair (i, i+dh/2) rotates by pos*theta^(-2i/dh) */
} bc_model_config;

/* Device pointers to one layer's weights, all bf16, [out, in] row-major.
 * w_qkv     [(Hq + 2*Hkv)*dh, h]: rows of the Hq query heads, then the Hkv key
 *           heads, then the Hkv value heads, each head's dh rows contiguous.
 * w_o       [h, Hq*dh]
 * w_gate_up [2*F, h]: rows 0..F-1 gate, rows F..2F-1 up;
 *           ffn(x) = w_down (silu(gate x) * (up x)).
 * w_down    [h, F]
 * attn_norm, ffn_norm [h]: RMSNorm gains.
 * b_qkv     [(Hq + 2*Hkv)*dh] or NULL: bias of the Q/K/V projection, same row
 *           order as w_qkv, added before RoPE (Qwen2-style layers, e.g.
 *           Dream-7B); NULL for none.
 * The weights are referenced, not copied, and must outlive the model. */
typedef struct {
  const void* w_qkv;
  const void* w_o;
  const void* w_gate_up;
  const void* w_down;
  const void* attn_norm;
  const void* ffn_norm;
  const void* b_qkv;
} bc_layer_weights;

typedef struct bc_model bc_model;

/* Creates a model over caller-owned weights (`layers` has cfg->n_layers
 * entries; the array itself is copied).  cache_capacity >= 1 is the number of
 * prefixes the KV store H holds before FIFO eviction (Appendix C).  Host only:
 * enqueues nothing. */
bc_status bc_model_create(const bc_model_config* cfg, const bc_layer_weights* layers,
                          int cache_capacity, bc_model** out);
/* Destroys the model and its table.  Cache memory stays the caller's. */
bc_status bc_model_destroy(bc_model* model);

/* --------------------------------------------------------- prefix cache */

/* Device bytes of one cache entry for a prefix of m tokens caching the first
 * n_layers_to_cache (Lc) layers, 0 <= Lc <= L.  Layout (byte offsets from the
 * entry base, see bc_cache_offset):
 *   KV$  [Lc][2 (K, V)][Hkv][m][dh] bf16, post-RoPE prefix keys and values of
 *        the prefix-only forward (KV$_l of Eq. 4);
 *   H$   at the next 256-byte boundary: [min(Lc+1, L)][m][h] fp32, the prefix
 *        residual entering layers 0..min(Lc, L-1) (H$[0] is the input itself).
 * Returns 0 for invalid arguments. */
size_t bc_prefix_cache_bytes(const bc_model* model, int m, int n_layers_to_cache);

/* Byte offset inside such an entry of element (layer, part, head, pos, dim):
 * part 0 = K, 1 = V (head < Hkv, dim < dh, layer < Lc), 2 = H$ (head ignored,
 * dim < h, layer <= min(Lc, L-1)).  Returns (size_t)-1 when out of range. */
size_t bc_cache_offset(const bc_model* model, int m, int n_layers_to_cache, int layer, int part,
                       int head, int pos, int dim);

/* Device workspace bytes that bc_prefix_populate needs for a prefix of m tokens. */
size_t bc_populate_workspace_bytes(const bc_model* model, int m);

/* Populate on a miss (Sec. 5.2): runs the prefix-only forward x_pref = p at
 * positions 0..m-1 through layers 0..Lc-1, writes the entry into cache_mem
 * (layout above) and inserts `key` into the store.  With Lc = L the residual
 * after the last layer has no H$ slot, so that layer computes its K/V only
 * (norm and Q/K/V projection).  If the store is full the
 * oldest entry is evicted first: *evicted = 1 and *evicted_key = its key (the
 * caller may free that entry's memory once `stream` has passed this call);
 * otherwise *evicted = 0, *evicted_key = 0 (either output may be NULL).
 *   x_prefix   device bf16 [m, h], m >= 1
 *   cache_mem  device, >= bc_prefix_cache_bytes(model, m, Lc) bytes, 256-byte
 *              aligned, referenced by the entry until it is invalidated or
 *              evicted
 *   workspace  device, >= bc_populate_workspace_bytes(model, m) bytes, free for
 *              reuse once `stream` has passed this call
 * Errors: BC_E_STATE if `key` is already cached (invalidate it first),
 * BC_E_INVALID for bad sizes or pointers, BC_E_HIP if a launch fails (the key
 * is then not inserted). */
bc_status bc_prefix_populate(bc_model* model, uint64_t key, const void* x_prefix, int m,
                             int n_layers_to_cache, void* cache_mem, size_t cache_bytes,
                             void* workspace, size_t ws_bytes, void* stream,
                             uint64_t* evicted_key, int* evicted);

/* Looks up `key` in the store (the paper's O(1) hit test).  On a hit writes the
 * entry's m and Lc (either pointer may be NULL) and returns BC_OK; on a miss
 * returns BC_E_NOT_FOUND. */
bc_status bc_prefix_lookup(const bc_model* model, uint64_t key, int* m_out, int* n_layers_out);

/* Removes `key` from the store (BC_E_NOT_FOUND if absent).  The entry's memory
 * returns to the caller once work already enqueued on it has completed. */
bc_status bc_prefix_invalidate(bc_model* model, uint64_t key);

/* Writes up to max_keys cached keys, oldest first (the FIFO eviction order),
 * and their total count to *n_out. */
bc_status bc_cache_keys(const bc_model* model, uint64_t* keys, int max_keys, int* n_out);

/* Prefix key k = h(p) of Appendix C: 64-bit xxHash (XXH64, seed 0) over the
 * token IDs as little-endian int32.  Host only. */
uint64_t bc_prefix_key(const int32_t* token_ids, size_t n);

/* ------------------------------------------------------------------ step */

/* Device workspace bytes that bc_step_forward needs. */
size_t bc_step_workspace_bytes(const bc_model* model, int m, int B, int n_s, int d);

/* Work accounting of a step, host only, exactly what bc_step_forward launches:
 * for each layer l (arrays of n_layers ints, any may be NULL)
 *   rows[l]      token rows projected by layer l: B*n_s if l < d, B*(m+n_s) otherwise
 *   pos_base[l]  RoPE position of the first projected row of a request:
 *                m for l < d (suffix positions m..m+n_s-1), 0 otherwise
 *   reads_kv[l]  1 if layer l reads the cached KV$_l (l < d), else 0
 * and *reads_h (may be NULL) = the H$ layer re-entered at d (d < L), or -1.
 * When d < L the last layer projects every row but runs attention, the O
 * projection and the FFN over the B*n_s suffix rows only: the prefix rows'
 * outputs of the last layer are never read, their K/V are. */
bc_status bc_step_plan(const bc_model* model, int m, int B, int n_s, int d, int* rows,
                       int* pos_base, int* reads_kv, int* reads_h);

/* One denoising-step forward of B requests sharing the cached prefix `key`
 * (Eq. 4 for layers l < d, the refresh case of Eq. 5 for l >= d).
 *   x_suffix  device bf16 [B, n_s, h]: each request's non-shared rows z_t, at
 *             positions m..m+n_s-1
 *   d         reuse depth, 0 <= d <= L and d <= the entry's Lc; d = 0 is the
 *             un-cached forward, d = L reuses the cache in every layer
 *   out       device fp32 [B, n_s, h]: final residual of the suffix rows (no
 *             final norm, no LM head)
 *   workspace device, >= bc_step_workspace_bytes(model, m, B, n_s, d) bytes
 * Requests never attend to each other.  Errors: BC_E_NOT_FOUND on a miss,
 * BC_E_INVALID for bad sizes, pointers or d. */
bc_status bc_step_forward(bc_model* model, uint64_t key, const void* x_suffix, int B, int n_s,
                          int d, float* out, void* workspace, size_t ws_bytes, void* stream);

/* ----------------------------------------------- batches of several prefixes
 *
 * In multi-tenant serving (Sec. 6.5) the requests of one batch come with
 * different shared prefixes: each request's prefix p is looked up in H under
 * k = h(p) (Sec. 5.2).  A batch is given as n_groups groups: group g holds
 * counts[g] consecutive requests of x_suffix that share the cached prefix
 * keys[g] (its own m_g).  Every request is computed exactly as in a
 * single-prefix step over its own prefix (requests never attend to each
 * other); one reuse depth d applies to the whole batch. */

/* Device workspace bytes that bc_step_forward_multi needs; 0 if an argument
 * is invalid or a key is not cached. */
size_t bc_step_multi_workspace_bytes(const bc_model* model, const uint64_t* keys, const int* counts,
                                     int n_groups, int n_s, int d);

/* One denoising step (Eq. 4 for l < d, refresh case of Eq. 5 for l >= d) of a
 * batch over several cached prefixes.
 *   keys, counts  host arrays of n_groups entries, 1 <= n_groups <= 4096,
 *                 counts[g] >= 1; a key may appear in several groups
 *   x_suffix      device bf16 [B, n_s, h], B = sum of counts; request i of
 *                 group g is row block (counts[0] + ... + counts[g-1] + i);
 *                 its positions are m_g..m_g+n_s-1
 *   d             0 <= d <= L and d <= every entry's Lc
 *   out           device fp32 [B, n_s, h], same request order
 *   workspace     device, >= bc_step_multi_workspace_bytes(...) bytes
 * The Q/K/V projection and the attention run once per group, every other
 * kernel once over the whole batch.  Errors: BC_E_NOT_FOUND if any key is not
 * cached, BC_E_INVALID for bad sizes, pointers or d. */
bc_status bc_step_forward_multi(bc_model* model, const uint64_t* keys, const int* counts,
                                int n_groups, const void* x_suffix, int n_s, int d, float* out,
                                void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------- deep-layer reuse (Eq. 5)
 *
 * Within one request the deep layers (l >= d) need not recompute the prefix
 * at every step (Sec. 5.2, Eq. 5): at a refresh step, (t - 1) mod delta == 0
 * with t the 1-based step index and delta the refresh interval, they
 * recompute it (exactly bc_step_forward); at every other step they reuse the
 * prefix K/V that the request's last refresh step computed, so the whole step
 * runs on the suffix rows only.  Those K/V live in a caller-owned "deep
 * store", one per batch of requests that step together. */

/* 1 if step t (1-based) of a request is a refresh step for refresh interval
 * delta, i.e. (t - 1) mod delta == 0; 0 if it reuses; -1 if t < 1 or
 * delta < 1.  Host only. */
int bc_is_refresh_step(int t, int delta);

enum {
  BC_DEEP_REFRESH = 0, /* first case of Eq. 5: deep layers recompute the prefix */
  BC_DEEP_REUSE = 1    /* second case: deep layers attend over the stored prefix K/V */
};

/* Device bytes of the deep store of a batch of B requests with n_s suffix rows
 * each over a prefix of m tokens at reuse depth d.  Layout: for each deep
 * layer l = d..L-1, K then V, each [B][Hkv][m + n_s][dh] bf16 (post-RoPE, the
 * refresh step's K/V of every row of the request; reuse steps read rows
 * 0..m-1), then a 256-byte header that the refresh step writes (its tag, see
 * bc_step_forward_deep).  Returns 0 for invalid arguments and for d = L (no
 * deep layers). */
size_t bc_deep_store_bytes(const bc_model* model, int m, int B, int n_s, int d);

/* Byte offset inside a deep store of element (layer, part, req, head, pos,
 * dim): d <= layer < L, part 0 = K / 1 = V, req < B, head < Hkv,
 * pos < m + n_s, dim < dh.  Returns (size_t)-1 when out of range. */
size_t bc_deep_store_offset(const bc_model* model, int m, int B, int n_s, int d, int layer,
                            int part, int req, int head, int pos, int dim);

/* Drops the tag of the deep store at `deep_store` (see bc_step_forward_deep),
 * so that a reuse step on it is refused until a refresh step writes it again.
 * Call it whenever memory at that address is newly allocated or put to other
 * use: the tag is keyed by address, and allocators hand addresses out again.
 * Returns BC_OK whether or not the address was tagged.  Host only. */
bc_status bc_deep_store_reset(bc_model* model, const void* deep_store);

/* One denoising step of B requests sharing the cached prefix `key`, with the
 * deep layers in either case of Eq. 5.
 *   mode BC_DEEP_REFRESH: the same computation and output as bc_step_forward;
 *        if deep_store is not NULL, the deep layers' K/V of every row are
 *        written into it (layout above) and the store is tagged with
 *        (key, m, B, n_s, d).  deep_store may be NULL (nothing is stored).
 *   mode BC_DEEP_REUSE: every layer runs on the suffix rows only (positions
 *        m..m+n_s-1).  Layers l < d attend over [KV$_l ; own suffix K/V]
 *        (Eq. 4), layers l >= d over [request b's prefix rows of the deep
 *        store ; own suffix K/V].  The store is only read.  The store must
 *        carry the tag of a refresh step with the same key, m, B, n_s and d
 *        (else BC_E_STATE); request b of this call must be request b of that
 *        refresh.  The library keeps the tag on the host, keyed by the store's
 *        address (bc_deep_store_reset drops it).  The refresh also writes the
 *        tag, with a number unique to that refresh, into the store's last 256
 *        bytes; the reuse step compares them on the device and, if they
 *        differ (the memory was overwritten since), writes NaN to every
 *        element of `out` (no error code: the check runs on the stream).
 *        Memory overwritten only inside the K/V blocks goes undetected.
 *   At d = L there are no deep layers: both modes equal bc_step_forward and
 *   deep_store is ignored (may be NULL).
 *   deep_store  device, >= bc_deep_store_bytes(model, m, B, n_s, d) bytes,
 *               256-byte aligned, caller-owned
 *   workspace   device, >= bc_step_workspace_bytes(model, m, B, n_s, d) bytes
 *               (a reuse step needs no more than
 *               bc_step_workspace_bytes(model, m, B, n_s, L))
 * Other arguments and errors as bc_step_forward; a refresh of a batch is for
 * all its requests at once (per-request schedules need separate batches), and
 * the batch shares one prefix (a multi-prefix batch keeps a store per prefix
 * group by stepping each group as its own batch). */
bc_status bc_step_forward_deep(bc_model* model, uint64_t key, const void* x_suffix, int B,
                               int n_s, int d, int mode, void* deep_store, size_t store_bytes,
                               float* out, void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------- shared-prefix profiling
 *
 * Offline profiling (Sec. 5.1) measures, for a request with prefix p and
 * suffix z, the KV similarity of Eq. 3 at the first step for every layer:
 *   sim_l = cos(flatten(KV$_l), flatten(KV^ref_{l,1}))
 * where KV$_l are the cached prefix-only KVs and KV^ref_{l,1} the prefix
 * rows' KVs of the un-cached forward of (p, z); K and V of every head and
 * position form one vector.  The shallow depth of the request is the largest
 * b with sim_l >= tau for every 1-based layer l <= b (Sec. 4.2), and the
 * lookup table T maps the shared-prefix ratio r = m / (m + n_s) to the mean b
 * of the profiled requests at that r. */

/* Device workspace bytes of bc_profile_similarity. */
size_t bc_profile_workspace_bytes(const bc_model* model, int m, int B, int n_s);

/* sim_l of B requests over the cached prefix `key`, which must cache all L
 * layers (n_layers_to_cache = L at populate).
 *   x_suffix  device bf16 [B, n_s, h]: the requests' non-shared rows at the
 *             first step (positions m..m+n_s-1)
 *   sims      device fp64 [B, L]: sims[b*L + l] = sim of 0-based layer l
 *   workspace device, >= bc_profile_workspace_bytes(model, m, B, n_s) bytes
 * Runs the un-cached step (d = 0) storing every layer's K/V, then one
 * HBM-bound reduction per layer (fp32 lane sums, fp64 across lanes and
 * workgroups, fixed order: results repeat bit for bit).  Errors as
 * bc_step_forward; BC_E_INVALID if the entry caches fewer than L layers. */
bc_status bc_profile_similarity(bc_model* model, uint64_t key, const void* x_suffix, int B, int n_s,
                                double* sims, void* workspace, size_t ws_bytes, void* stream);

/* Device workspace bytes of bc_cosine_similarity (0 if n is invalid). */
size_t bc_cosine_workspace_bytes(long n);

/* *out = cos(a, b) of two bf16 device vectors of n elements (n a positive
 * multiple of 8, 16-byte aligned), into device fp64 memory, with the same
 * reduction as bc_profile_similarity.  A zero vector gives NaN. */
bc_status bc_cosine_similarity(const void* a, const void* b, long n, double* out, void* workspace,
                               size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * result as bc_cosine_similarity, bit for bit (same kernels, same reduction
 * order), with no workspace argument.  The reduction's partial sums go to a
 * static 4 MiB device array of the library, one per GPU it runs on, held
 * until the process ends; this call allocates nothing and enqueues only the
 * two reduction kernels.  n is a positive multiple of 8 of at most
 * 130,146,304 elements (15,887 workgroup partials of 33 fp64 values); a
 * larger n returns BC_E_CAPACITY before anything is enqueued.  Every call on a GPU shares that GPU's array: calls that
 * overlap on one GPU (other streams, other threads) race and must be
 * serialized by the caller.  Nothing carries over between calls.
 * Other arguments and errors as bc_cosine_similarity. */
bc_status bc_cosine_similarity_noalloc(const void* a, const void* b, long n, double* out,
                                       void* stream);

/* The shallow depth b of Sec. 4.2: the number of leading entries of
 * sims[0..n_layers) that are >= tau (0..n_layers); -1 for bad arguments.
 * Host only. */
int bc_shallow_depth(const double* sims, int n_layers, double tau);

/* Table T (Sec. 5.1) over ratio buckets r = k / n_buckets, k = 1..n_buckets:
 * request i (ratio ratios[i], which must be a bucket value, and profiled
 * depth depths[i] >= 0) falls into bucket k; table[k] = floor(mean depth of
 * bucket k), or -1 for a bucket without requests; table[0] = -1.  table has
 * n_buckets + 1 entries.  Host only. */
bc_status bc_build_depth_table(const double* ratios, const int* depths, int n, int n_buckets,
                               int* table);

/* d for a request of shared-prefix ratio r: table[k] of the largest bucket
 * k <= r * n_buckets that has data (rounding down is the safe side, as b
 * grows with r); 0 if none; -1 for bad arguments.  Host only. */
int bc_depth_lookup(const int* table, int n_buckets, double r);

/* ------------------------------------------------------------ profiling */

/* Kernel classes of the step and of populate, for bc_profile_* below. */
enum {
  BC_K_RMSNORM = 0,     /* RMSNorm (both norms of a layer) */
  BC_K_QKV = 1,         /* fused Q/K/V projection + RoPE (+ cache write in populate) */
  BC_K_ATTN_SHARED = 2, /* attention over [cached prefix ; own suffix]: layers l < d,
                           and every layer of a reuse step */
  BC_K_ATTN_FULL = 3,   /* full attention of each request (layers l >= d, populate) */
  BC_K_OPROJ = 4,       /* output projection + residual add */
  BC_K_GATE_UP = 5,     /* gate/up projection + SwiGLU */
  BC_K_DOWN = 6,        /* down projection + residual add */
  BC_K_OTHER = 7,       /* RoPE table, input widening, suffix gather */
  BC_K_KVSIM = 8,       /* KV-similarity reduction of bc_profile_similarity */
  BC_K_TRANSITION = 9,  /* full residual at l = d: cached prefix residual broadcast to
                           every request, followed by its suffix rows */
  BC_K_COUNT = 10
};

/* Starts timing, with HIP events recorded on the launch stream around every
 * later launch of a class whose bit (1u << class) is set in kernel_mask.
 * Measurement only: the events add a small gap between kernels. */
bc_status bc_profile_begin(bc_model* model, unsigned kernel_mask);

/* Waits for the recorded events, writes per class the summed kernel time in
 * milliseconds (ms[BC_K_COUNT]) and the number of timed launches
 * (launches[BC_K_COUNT]), then stops timing.  Either array may be NULL. */
bc_status bc_profile_end(bc_model* model, double* ms, int* launches);

/* ------------------------------------------------------- attention only */

/* Shared-prefix bidirectional attention (Eq. 2 over [prefix ; own suffix], the
 * shallow-layer form of Eq. 4), one launch:
 *   out[b,j,i,:] = sum_t softmax_t(scale * q[b,j,i,:] . K_t) V_t
 * over the keys t of [k_pre[g] ; k_suf[b,g]] with g = j / (Hq/Hkv); no mask.
 *   q            bf16 [B, Hq, n_s, dh]
 *   k_pre, v_pre bf16 [Hkv, m, dh]   one copy shared by all B requests (m >= 0)
 *   k_suf, v_suf bf16 [B, Hkv, n_s, dh]
 *   out          fp32 [B, Hq, n_s, dh]
 * B, n_s >= 1; dh in {64, 128}; Hq % Hkv == 0.  Products use bf16 operands
 * with fp32 accumulation; the softmax is fp32 (probabilities are rounded to
 * bf16 for the P.V product). */
bc_status bc_shared_prefix_attention(const void* q, const void* k_pre, const void* v_pre,
                                     const void* k_suf, const void* v_suf, float* out, int B,
                                     int Hq, int Hkv, int m, int n_s, int dh, float scale,
                                     void* stream);

/* Attention over [each request's own prefix ; own suffix] (Eq. 2, the deep
 * layers of a reuse step, second case of Eq. 5), one launch:
 *   out[b,j,i,:] = sum_t softmax_t(scale * q[b,j,i,:] . K_t) V_t
 * over the keys t of [k_pre[b,g] ; k_suf[b,g]] with g = j / (Hq/Hkv); no mask.
 *   q            bf16 [B, Hq, n_s, dh]
 *   k_pre, v_pre bf16 [B, Hkv, m, dh]   request b's prefix K/V (m >= 0)
 *   k_suf, v_suf bf16 [B, Hkv, n_s, dh]
 *   out          fp32 [B, Hq, n_s, dh]
 * Sizes, precision and errors as bc_shared_prefix_attention. */
bc_status bc_request_prefix_attention(const void* q, const void* k_pre, const void* v_pre,
                                      const void* k_suf, const void* v_suf, float* out, int B,
                                      int Hq, int Hkv, int m, int n_s, int dh, float scale,
                                      void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BICACHE_H */
