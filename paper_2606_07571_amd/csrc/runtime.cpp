// Host runtime and C ABI of libbicache.so: argument validation, the KV store H
// with FIFO eviction, cache-entry, deep-store and workspace layouts, and the
// layer loops of populate (prefix-only forward), of the step at reuse depth d
// (refresh case of Eq. 5 for the deep layers) and of the reuse step (second
// case of Eq. 5).
//
// Every device buffer is the caller's; this file only carves caller-provided
// workspace into sub-buffers and enqueues kernels on the caller's stream.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <new>
#include <string>
#include <atomic>
#include <mutex>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "../../include/bicache.h"
#include "cache_table.hpp"
#include "kernels.hpp"

// HIP-event timing of selected kernel classes (bc_profile_*).
struct Profiler {
  unsigned mask = 0;
  std::vector<hipEvent_t> pool;  // reused across sessions, destroyed with the model
  size_t used = 0;
  struct Rec {
    int kind;
    size_t start, stop;
  };
  std::vector<Rec> recs;
};

// What the last refresh step wrote into a deep store (keyed by its address):
// a reuse step must match it.  `nonce` is unique to that refresh (process-wide
// counter); the refresh also writes the tag into the store's header, and a
// reuse step compares the two on the device (deep_header_words).
struct DeepTag {
  uint64_t key;
  int m, B, n_s, d;
  uint64_t nonce;
};
static std::atomic<uint64_t> g_deep_nonce{1};
constexpr uint64_t kDeepMagic = 0x3130504545444342ull;  // "BCDEEP01"
static bc::DeepHeader deep_header_words(const DeepTag& t) {
  bc::DeepHeader h{};
  h.w[0] = kDeepMagic;
  h.w[1] = t.key;
  h.w[2] = (uint64_t)(uint32_t)t.m | (uint64_t)(uint32_t)t.B << 32;
  h.w[3] = (uint64_t)(uint32_t)t.n_s | (uint64_t)(uint32_t)t.d << 32;
  h.w[4] = t.nonce;
  h.w[5] = ~(t.key ^ t.nonce);
  return h;
}

struct bc_model {
  bc_model_config cfg;
  std::vector<bc_layer_weights> layers;
  bc::CacheTable table;
  Profiler prof;
  std::unordered_map<uintptr_t, DeepTag> deep_tags;
  bc_model(const bc_model_config& c, const bc_layer_weights* l, int cap)
      : cfg(c), layers(l, l + c.n_layers), table(cap) {}
  ~bc_model() {
    for (hipEvent_t e : prof.pool) (void)hipEventDestroy(e);
  }
};

namespace {

// The calling thread's last error message; a fixed buffer, so that reporting
// a failed host allocation needs no allocation itself.
thread_local char g_err[512];

bc_status fail(bc_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

bc_status ok() {
  g_err[0] = 0;
  return BC_OK;
}

// Status of a C++ exception caught at the boundary (none crosses it): a failed
// host allocation is BC_E_OOM, anything else BC_E_INVALID.
bc_status host_exception() {
  try {
    throw;
  } catch (const std::bad_alloc&) {
    return fail(BC_E_OOM, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(BC_E_INVALID, "host error: %s", e.what());
  } catch (...) {
    return fail(BC_E_INVALID, "unknown host error");
  }
}

// Handles of the models that exist: a call with a destroyed or unknown handle
// is refused (BC_E_INVALID) instead of reading freed memory.
std::mutex g_models_mu;
std::unordered_set<const bc_model*> g_models;

bool live(const bc_model* m) {
  if (!m) return false;
  std::lock_guard<std::mutex> lk(g_models_mu);
  return g_models.count(m) != 0;
}

constexpr size_t kAlign = 256;
constexpr uintptr_t kVecAlign = 16;  // kernels move 16-byte vectors
bool misaligned(const void* p) { return ((uintptr_t)p % kVecAlign) != 0; }
constexpr int kMaxGroups = 4096;  // prefix groups in one batch
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Sub-buffer plan of a workspace.  All offsets are 256-byte aligned.
struct Plan {
  size_t cos = 0, sin = 0, xn = 0, q = 0, k = 0, v = 0, ao = 0, act = 0, R = 0, total = 0;
};

struct Bump {
  size_t at = 0;
  size_t take(size_t bytes) {
    const size_t o = at;
    at = align_up(at + bytes);
    return o;
  }
};

// rows: token rows a layer processes at most; n_pos: RoPE table positions;
// with_kv: K/V live in the workspace (step) rather than in the cache (populate);
// resid_rows: rows of the fp32 residual kept in the workspace (0 = none).
Plan make_plan(const bc_model_config& c, long rows, long n_pos, bool with_kv, long resid_rows) {
  Plan p;
  Bump b;
  const long hd = (long)c.n_heads * c.head_dim, kvd = (long)c.n_kv_heads * c.head_dim;
  p.cos = b.take(n_pos * (c.head_dim / 2) * 4);
  p.sin = b.take(n_pos * (c.head_dim / 2) * 4);
  p.xn = b.take(rows * c.hidden * 2);
  p.q = b.take(rows * hd * 2);
  if (with_kv) {
    p.k = b.take(rows * kvd * 2);
    p.v = b.take(rows * kvd * 2);
  }
  p.ao = b.take(rows * hd * 2);
  p.act = b.take(rows * (long)c.ffn * 2);
  if (resid_rows) p.R = b.take(resid_rows * c.hidden * 4);
  p.total = b.at;
  return p;
}

// Cache entry layout: KV$ [Lc][2][Hkv][m][dh] bf16, then H$ [nH][m][h] fp32.
struct EntryLayout {
  size_t kv_layer = 0;  // bytes of one layer's K or V block
  size_t h_off = 0, h_layer = 0, total = 0;
  int n_h = 0;
};

EntryLayout entry_layout(const bc_model_config& c, int m, int Lc) {
  EntryLayout e;
  e.kv_layer = (size_t)c.n_kv_heads * m * c.head_dim * 2;
  e.h_off = align_up((size_t)Lc * 2 * e.kv_layer);
  e.n_h = Lc + 1 < c.n_layers ? Lc + 1 : c.n_layers;
  e.h_layer = (size_t)m * c.hidden * 4;
  e.total = e.h_off + (size_t)e.n_h * e.h_layer;
  return e;
}

// Deep store of a batch: for each deep layer l in [d, L), K then V, each
// [B][Hkv][N][dh] bf16 with N = m + n_s (the refresh step's K/V of every row;
// reuse steps read rows 0..m-1), then a 256-byte header (the refresh's tag).
// Every block is a multiple of 256 bytes.
constexpr size_t kDeepHeaderBytes = 256;
struct DeepLayout {
  size_t part = 0;    // bytes of one layer's K or V block
  size_t header = 0;  // offset of the header
  size_t total = 0;
  long sb = 0, sh = 0;  // request and head strides (elements)
};

DeepLayout deep_layout(const bc_model_config& c, int m, int B, int n_s, int d) {
  DeepLayout dl;
  const long N = (long)m + n_s;
  dl.sh = N * c.head_dim;
  dl.sb = (long)c.n_kv_heads * dl.sh;
  dl.part = (size_t)B * dl.sb * 2;
  if (d >= c.n_layers) return dl;  // no deep layers: no store
  dl.header = align_up((size_t)(c.n_layers - d) * 2 * dl.part);
  dl.total = dl.header + kDeepHeaderBytes;
  return dl;
}

bool config_ok(const bc_model_config& c, std::string* why) {
  char buf[256];
  auto bad = [&](const char* s) {
    snprintf(buf, sizeof buf, "invalid model config: %s", s);
    *why = buf;
    return false;
  };
  if (c.n_layers < 1) return bad("n_layers must be >= 1");
  if (c.hidden < 64 || c.hidden % 64 || c.hidden > 8192) return bad("hidden must be a multiple of 64 in [64, 8192]");
  if (c.head_dim != 64 && c.head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c.n_heads < 1 || c.n_kv_heads < 1 || c.n_heads % c.n_kv_heads)
    return bad("n_heads must be a positive multiple of n_kv_heads");
  if (c.ffn < 64 || c.ffn % 64) return bad("ffn must be a positive multiple of 64");
  if (!(c.rms_eps >= 0.f) || !(c.rope_theta > 0.f)) return bad("rms_eps >= 0 and rope_theta > 0 required");
  return true;
}

#define BC_HIP(expr)                                                                 \
  do {                                                                               \
    hipError_t e_ = (expr);                                                          \
    if (e_ != hipSuccess)                                                            \
      return fail(BC_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));          \
  } while (0)

// Records an event on `s` if class `kind` is being timed; returns its pool
// index in *idx (or SIZE_MAX when not timing).
hipError_t prof_mark(bc_model* mdl, int kind, hipStream_t s, size_t* idx) {
  *idx = SIZE_MAX;
  Profiler& p = mdl->prof;
  if (!(p.mask & (1u << kind))) return hipSuccess;
  if (p.used == p.pool.size()) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    p.pool.push_back(e);
  }
  *idx = p.used++;
  return hipEventRecord(p.pool[*idx], s);
}

// Launch `expr` (a hipError_t expression), timed as class `kind` when enabled.
#define BC_LAUNCH(mdl, kind, s, expr)                                             \
  do {                                                                           \
    size_t i0_, i1_;                                                             \
    BC_HIP(prof_mark(mdl, kind, s, &i0_));                                       \
    BC_HIP(expr);                                                                \
    BC_HIP(prof_mark(mdl, kind, s, &i1_));                                       \
    if (i0_ != SIZE_MAX) mdl->prof.recs.push_back({kind, i0_, i1_});             \
  } while (0)

// One transformer layer over the token rows held in the fp32 residual R.  The
// rows form segments; segment i covers rows [row0, row0 + n_req*n_seq), row
// row0 + r being token t = r % n_seq of its request r / n_seq at RoPE position
// pos0 + t.  A segment's own K/V are written to k_dst/v_dst (element (req,
// head, t, dim) at req*kv_sb + head*kv_sh + t*dh + dim) and each of its
// requests attends over [kp/vp (m_pre prefix rows, may be 0) ; its own n_seq
// keys]; the prefix is shared by the segment's requests when kp_sb == 0, else
// request r's starts at kp + r*kp_sb (head stride kp_sh, 0 = m_pre*dh).
// Normalisation and the O / FFN GEMMs run once over all rows (rows are
// independent there); the Q/K/V projection and the attention run per segment.
struct Seg {
  long row0;
  int n_req, n_seq, pos0;
  const void* kp;
  const void* vp;
  int m_pre;
  void* k_dst;
  void* v_dst;
  long kv_sb, kv_sh;
  long kp_sb = 0, kp_sh = 0;
};

// How much of a layer runs.  kAll: the whole layer over lc.rows rows.
// kKvOnly: norm and Q/K/V projection only (a populate's last layer whose
// output residual no cache slot keeps).  kSuffixOut: the last layer of a step
// whose deep layers run over every row.  Only the suffix rows' outputs are
// ever read there (the step returns them; nothing reads the prefix rows'
// hidden states after the last layer), so once Q/K/V of every row are
// projected (the suffix rows attend to the recomputed prefix K/V, Eq. 5 first
// case) the suffix rows of the residual move to lc.out, and attention, the O
// projection and the FFN run over those rows alone.  Per row the arithmetic
// is that of kAll: the attention walks each request's own prefix rows then its
// suffix rows, the same key tiles in the same order as the walk over all N
// rows whenever m is a multiple of the 64-key tile.
enum class LayerPart { kAll, kKvOnly, kSuffixOut };

struct LayerCall {
  float* R;
  long rows;
  const Seg* segs;
  int n_segs;
  // kSuffixOut: the suffix rows' residual [B][n_s][h]; segment i's requests
  // start at request first[i]
  float* out = nullptr;
  const int* first = nullptr;
  int B = 0, n_s = 0;
};

bc_status run_layer(bc_model* mdl, int l, const LayerCall& lc, char* ws, const Plan& p,
                    hipStream_t s, LayerPart part = LayerPart::kAll) {
  const bc_model_config& c = mdl->cfg;
  const bc_layer_weights& w = mdl->layers[l];
  const int h = c.hidden, Hq = c.n_heads, Hkv = c.n_kv_heads, dh = c.head_dim, F = c.ffn;
  const int hd = Hq * dh;
  const bool sfx = part == LayerPart::kSuffixOut;
  uint16_t* xn = (uint16_t*)(ws + p.xn);  // bf16 bits
  uint16_t* q = (uint16_t*)(ws + p.q);
  uint16_t* ao = (uint16_t*)(ws + p.ao);
  void* act = ws + p.act;
  const float* cos_t = (const float*)(ws + p.cos);
  const float* sin_t = (const float*)(ws + p.sin);

  BC_LAUNCH(mdl, BC_K_RMSNORM, s, bc::rmsnorm(lc.R, w.attn_norm, xn, (int)lc.rows, h, c.rms_eps, s));
  for (int i = 0; i < lc.n_segs; ++i) {
    const Seg& g = lc.segs[i];
    const int N = g.n_seq;
    uint16_t* qg = q + g.row0 * hd;
    bc::QkvOut qo{qg, g.k_dst, g.v_dst, (long)Hq * N * dh, (long)N * dh,
                  g.kv_sb, g.kv_sh, g.kv_sb, g.kv_sh, w.b_qkv};
    BC_LAUNCH(mdl, BC_K_QKV, s,
              bc::gemm_qkv_rope(xn + g.row0 * h, h, w.w_qkv, h, g.n_req * N, h, Hq, Hkv, dh, N, g.pos0,
                                cos_t, sin_t, qo, s));
    if (part == LayerPart::kKvOnly) continue;
    bc::AttnArgs a{};
    a.q_sb = (long)Hq * N * dh;
    a.q_sh = (long)N * dh;
    a.q_sr = dh;
    a.s_sb = g.kv_sb;
    a.s_sh = g.kv_sh;
    a.s_sr = dh;
    a.o_sh = dh;  // token-major [req, t, head, dim]: the O projection's A operand
    a.o_sr = hd;
    a.B = g.n_req;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.dh = dh;
    a.scale = 1.f / sqrtf((float)dh);
    a.out_f32 = 0;
    if (sfx) {
      const int m = N - lc.n_s;
      BC_LAUNCH(mdl, BC_K_OTHER, s,
                bc::gather_suffix(lc.R + g.row0 * h, lc.out + (long)lc.first[i] * lc.n_s * h, g.n_req, m,
                                  lc.n_s, h, s));
      a.q = qg + (long)m * dh;  // the suffix query rows of every (request, head)
      a.kp = g.k_dst;           // each request's own prefix rows 0..m-1
      a.vp = g.v_dst;
      a.p_sb = g.kv_sb;
      a.p_sh = g.kv_sh;
      a.ks = (const uint16_t*)g.k_dst + (long)m * dh;   // and its suffix rows m..N-1
      a.vs = (const uint16_t*)g.v_dst + (long)m * dh;
      a.out = ao + (long)lc.first[i] * lc.n_s * hd;
      a.o_sb = (long)lc.n_s * hd;
      a.m = m;
      a.n_s = lc.n_s;
      BC_LAUNCH(mdl, BC_K_ATTN_FULL, s, bc::attention(a, s));
    } else {
      a.q = qg;
      a.kp = g.kp;
      a.vp = g.vp;
      a.p_sb = g.kp_sb;
      a.p_sh = g.kp_sh ? g.kp_sh : (long)g.m_pre * dh;
      a.ks = g.k_dst;
      a.vs = g.v_dst;
      a.out = ao + g.row0 * hd;
      a.o_sb = (long)N * hd;
      a.m = g.m_pre;
      a.n_s = N;
      BC_LAUNCH(mdl, g.m_pre > 0 ? BC_K_ATTN_SHARED : BC_K_ATTN_FULL, s, bc::attention(a, s));
    }
  }
  if (part == LayerPart::kKvOnly) return BC_OK;
  float* R = sfx ? lc.out : lc.R;
  const int rows = sfx ? lc.B * lc.n_s : (int)lc.rows;
  BC_LAUNCH(mdl, BC_K_OPROJ, s, bc::gemm_residual(ao, hd, w.w_o, hd, rows, h, hd, R, h, s));
  BC_LAUNCH(mdl, BC_K_RMSNORM, s, bc::rmsnorm(R, w.ffn_norm, xn, rows, h, c.rms_eps, s));
  BC_LAUNCH(mdl, BC_K_GATE_UP, s, bc::gemm_swiglu(xn, h, w.w_gate_up, h, rows, F, h, act, s));
  BC_LAUNCH(mdl, BC_K_DOWN, s, bc::gemm_residual(act, F, w.w_down, F, rows, h, F, R, h, s));
  return BC_OK;
}

bool step_shape_ok(const bc_model_config& c, int m, int B, int n_s, int d, std::string* why) {
  char buf[256];
  if (m < 1 || B < 1 || n_s < 1) {
    snprintf(buf, sizeof buf, "m, B and n_s must be >= 1 (got m=%d B=%d n_s=%d)", m, B, n_s);
    *why = buf;
    return false;
  }
  if (d < 0 || d > c.n_layers) {
    snprintf(buf, sizeof buf, "reuse depth d=%d outside [0, L=%d]", d, c.n_layers);
    *why = buf;
    return false;
  }
  const long N = (long)m + n_s;
  const long rows = (long)B * N;
  const long widest = c.ffn > (long)c.n_heads * c.head_dim ? c.ffn : (long)c.n_heads * c.head_dim;
  if (N > INT_MAX / 2 || rows > INT_MAX / 2 || rows * (widest > c.hidden ? widest : c.hidden) > (1L << 40) ||
      rows * (long)c.hidden / 4 > (long)INT_MAX) {
    snprintf(buf, sizeof buf, "step too large (B=%d, m+n_s=%ld)", B, N);
    *why = buf;
    return false;
  }
  return true;
}


// A group of a batch: `count` consecutive requests over the cached prefix
// `key` (one group unless the batch spans several prefixes).
struct Group {
  uint64_t key;
  int count;
};

// The step, for every kind: mode BC_DEEP_REFRESH: layers l < d suffix-only
// over KV$_l, layers l >= d recompute the prefix from H$_d (their K/V of every
// row go to `store` when it is non-null, else to the workspace).
// BC_DEEP_REUSE: every layer suffix-only, deep layers over the request's
// prefix rows in `store`.  The deep store is for single-prefix batches only.
// Work layout with several groups: the shallow residual is `out` [B][n_s][h]
// (group g's requests at rows first_g*n_s...); the deep residual, Q/K/V and
// attention output hold the groups one after another, group g's requests
// with N_g = m_g + n_s rows each.
bc_status step_impl(bc_model* model, const Group* groups, int n_groups, const void* x_suffix,
                    int n_s, int d, int mode, void* store, size_t store_bytes, float* out,
                    void* workspace, size_t ws_bytes, void* stream) {
  if (!live(model) || !groups || !x_suffix || !out || !workspace) return fail(BC_E_INVALID, "null argument");
  if (misaligned(x_suffix) || misaligned(out)) return fail(BC_E_INVALID, "x_suffix and out must be 16-byte aligned");
  if (mode != BC_DEEP_REFRESH && mode != BC_DEEP_REUSE) return fail(BC_E_INVALID, "unknown deep mode %d", mode);
  if (n_groups < 1 || n_groups > kMaxGroups)
    return fail(BC_E_INVALID, "n_groups=%d outside [1, %d]", n_groups, kMaxGroups);
  const bc_model_config& c = model->cfg;
  const int L = c.n_layers;
  std::vector<const bc::CacheEntry*> ents(n_groups);
  long B = 0, full_rows = 0;
  int max_N = 0;
  std::string why;
  for (int g = 0; g < n_groups; ++g) {
    ents[g] = model->table.find(groups[g].key);
    if (!ents[g]) return fail(BC_E_NOT_FOUND, "key %016llx is not cached", (unsigned long long)groups[g].key);
    const int m = ents[g]->m;
    if (groups[g].count < 1) return fail(BC_E_INVALID, "group %d has count %d < 1", g, groups[g].count);
    if (!step_shape_ok(c, m, groups[g].count, n_s, d, &why)) return fail(BC_E_INVALID, "%s", why.c_str());
    if (d > ents[g]->n_layers)
      return fail(BC_E_INVALID, "reuse depth d=%d exceeds the %d cached layers of prefix %016llx", d,
                  ents[g]->n_layers, (unsigned long long)groups[g].key);
    B += groups[g].count;
    full_rows += (long)groups[g].count * (m + n_s);
    if (m + n_s > max_N) max_N = m + n_s;
  }
  // the elementwise kernels run one lane per 4 residual values on a 1-D grid
  if (B > INT_MAX / 2 || full_rows > INT_MAX / 2 || full_rows * (long)c.hidden / 4 > (long)INT_MAX)
    return fail(BC_E_INVALID, "step too large (B=%ld, %ld full rows)", B, full_rows);
  const bool full = mode == BC_DEEP_REFRESH && d < L;  // deep layers run over all rows
  const long rows_max = full ? full_rows : B * n_s;
  const Plan p = make_plan(c, rows_max, max_N, true, full ? full_rows : 0);
  if (ws_bytes < p.total) return fail(BC_E_INVALID, "workspace %zu < required %zu", ws_bytes, p.total);
  if ((uintptr_t)workspace % kAlign) return fail(BC_E_INVALID, "workspace must be 256-byte aligned");
  const bool use_store = d < L && (mode == BC_DEEP_REUSE || store);
  if (use_store && n_groups != 1)
    return fail(BC_E_INVALID, "deep-layer reuse (deep store) needs a single-prefix batch");
  const int m0 = ents[0]->m;
  const uint64_t key0 = groups[0].key;
  const DeepLayout dl = deep_layout(c, m0, (int)B, n_s, d);
  if (use_store) {
    if (!store) return fail(BC_E_INVALID, "a reuse step at d=%d < L needs the deep store", d);
    if (store_bytes < dl.total) return fail(BC_E_INVALID, "deep store %zu < required %zu", store_bytes, dl.total);
    if ((uintptr_t)store % kAlign) return fail(BC_E_INVALID, "deep store must be 256-byte aligned");
  }
  DeepTag reuse_tag{};
  if (use_store && mode == BC_DEEP_REUSE) {
    auto it = model->deep_tags.find((uintptr_t)store);
    if (it == model->deep_tags.end())
      return fail(BC_E_STATE, "no refresh step has written this deep store");
    const DeepTag& tg = it->second;
    reuse_tag = tg;
    if (tg.key != key0 || tg.m != m0 || tg.B != B || tg.n_s != n_s || tg.d != d)
      return fail(BC_E_STATE,
                  "deep store was refreshed for key %016llx m=%d B=%d n_s=%d d=%d, not key %016llx m=%d B=%ld n_s=%d d=%d",
                  (unsigned long long)tg.key, tg.m, tg.B, tg.n_s, tg.d, (unsigned long long)key0, m0, B, n_s, d);
  }

  // A refresh overwrites the store: its old tag no longer describes it, even if
  // a launch below fails part way.  The new tag is set once every launch is in.
  if (use_store && mode == BC_DEEP_REFRESH) model->deep_tags.erase((uintptr_t)store);

  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  char* st_mem = (char*)store;
  const int dh = c.head_dim, Hkv = c.n_kv_heads, h = c.hidden;
  const long kvd = (long)Hkv * dh;
  auto deep_k = [&](int l) { return st_mem + (size_t)(2 * (l - d)) * dl.part; };
  auto deep_v = [&](int l) { return st_mem + (size_t)(2 * (l - d) + 1) * dl.part; };
  std::vector<Seg> segs(n_groups);

  BC_LAUNCH(model, BC_K_OTHER, s, bc::rope_table((float*)(ws + p.cos), (float*)(ws + p.sin), max_N, dh, c.rope_theta, s));
  // suffix-only residual, kept in `out`
  BC_LAUNCH(model, BC_K_OTHER, s, bc::bf16_to_f32(x_suffix, out, B * n_s * h, s));
  const int n_suffix_layers = full ? d : L;
  for (int l = 0; l < n_suffix_layers; ++l) {
    long row0 = 0;
    for (int g = 0; g < n_groups; ++g) {
      const int m = ents[g]->m, cnt = groups[g].count;
      Seg& sg = segs[g];
      sg = Seg{row0, cnt, n_s, m, nullptr, nullptr, m,
               ws + p.k + row0 * kvd * 2, ws + p.v + row0 * kvd * 2, kvd * n_s, (long)n_s * dh};
      if (l < d) {  // Eq. 4: the shared KV$_l of the group's prefix
        const EntryLayout e = entry_layout(c, m, ents[g]->n_layers);
        const char* cm = (const char*)ents[g]->mem;
        sg.kp = cm + (size_t)(2 * l) * e.kv_layer;
        sg.vp = cm + (size_t)(2 * l + 1) * e.kv_layer;
      } else {      // second case of Eq. 5: this request's prefix K/V of the last refresh
        sg.kp = deep_k(l);
        sg.vp = deep_v(l);
        sg.kp_sb = dl.sb;
        sg.kp_sh = dl.sh;
      }
      row0 += (long)cnt * n_s;
    }
    LayerCall lc{out, B * n_s, segs.data(), n_groups};
    bc_status st = run_layer(model, l, lc, ws, p, s);
    if (st != BC_OK) return st;
  }
  if (full) {
    float* R = (float*)(ws + p.R);
    long row0 = 0, first = 0;
    for (int g = 0; g < n_groups; ++g) {
      const int m = ents[g]->m, cnt = groups[g].count;
      const EntryLayout e = entry_layout(c, m, ents[g]->n_layers);
      const float* hdp = (const float*)((const char*)ents[g]->mem + e.h_off + (size_t)d * e.h_layer);
      BC_LAUNCH(model, BC_K_TRANSITION, s,
                bc::build_full_residual(hdp, out + first * n_s * h, R + row0 * h, cnt, m, n_s, h, s));
      row0 += (long)cnt * (m + n_s);
      first += cnt;
    }
    std::vector<int> firsts(n_groups);
    for (int g = 0, f = 0; g < n_groups; f += groups[g].count, ++g) firsts[g] = f;
    for (int l = d; l < L; ++l) {
      row0 = 0;
      for (int g = 0; g < n_groups; ++g) {
        const int N = ents[g]->m + n_s, cnt = groups[g].count;
        void* kd = use_store ? (void*)deep_k(l) : (void*)(ws + p.k + row0 * kvd * 2);
        void* vd = use_store ? (void*)deep_v(l) : (void*)(ws + p.v + row0 * kvd * 2);
        segs[g] = Seg{row0, cnt, N, 0, nullptr, nullptr, 0, kd, vd, kvd * N, (long)N * dh};
        row0 += (long)cnt * N;
      }
      // the last layer also moves the suffix rows of the residual to `out`
      const LayerCall lc{R, full_rows, segs.data(), n_groups, out, firsts.data(), (int)B, n_s};
      bc_status st = run_layer(model, l, lc, ws, p, s, l + 1 < L ? LayerPart::kAll : LayerPart::kSuffixOut);
      if (st != BC_OK) return st;
    }
    if (use_store) {
      const DeepTag tg{key0, m0, (int)B, n_s, d, g_deep_nonce.fetch_add(1)};
      BC_LAUNCH(model, BC_K_OTHER, s,
                bc::deep_header_write((uint64_t*)(st_mem + dl.header), deep_header_words(tg), s));
      model->deep_tags[(uintptr_t)store] = tg;
    }
  } else if (use_store) {
    // a reuse step: if the store's header is not the tag of the refresh the
    // host recorded (the memory was overwritten since), every output is NaN
    BC_LAUNCH(model, BC_K_OTHER, s,
              bc::deep_header_check((const uint64_t*)(st_mem + dl.header), deep_header_words(reuse_tag),
                                    out, B * n_s * h, s));
  }
  return ok();
}

// Sizes of a step over groups, for the workspace functions (0 when invalid).
size_t step_workspace(const bc_model* model, const int* ms, const int* counts, int n_groups,
                      int n_s, int d) {
  const bc_model_config& c = model->cfg;
  long B = 0, full_rows = 0;
  int max_N = 0;
  std::string why;
  for (int g = 0; g < n_groups; ++g) {
    if (!step_shape_ok(c, ms[g], counts[g], n_s, d, &why)) return 0;
    B += counts[g];
    full_rows += (long)counts[g] * (ms[g] + n_s);
    if (ms[g] + n_s > max_N) max_N = ms[g] + n_s;
  }
  if (B > INT_MAX / 2 || full_rows > INT_MAX / 2) return 0;
  const bool full = d < c.n_layers;
  return make_plan(c, full ? full_rows : B * n_s, max_N, true, full ? full_rows : 0).total;
}

bc_status prefix_attention(const void* q, const void* k_pre, const void* v_pre, long pre_sb,
                           const void* k_suf, const void* v_suf, float* out, int B, int Hq,
                           int Hkv, int m, int n_s, int dh, float scale, void* stream) {
  if (!q || !k_suf || !v_suf || !out || (m > 0 && (!k_pre || !v_pre)))
    return fail(BC_E_INVALID, "null argument");
  if (misaligned(q) || misaligned(k_suf) || misaligned(v_suf) || misaligned(out) ||
      (m > 0 && (misaligned(k_pre) || misaligned(v_pre))))
    return fail(BC_E_INVALID, "q, k, v and out must be 16-byte aligned");
  if (B < 1 || n_s < 1 || m < 0) return fail(BC_E_INVALID, "B, n_s >= 1 and m >= 0 required");
  if (dh != 64 && dh != 128) return fail(BC_E_INVALID, "dh must be 64 or 128 (got %d)", dh);
  if (Hq < 1 || Hkv < 1 || Hq % Hkv) return fail(BC_E_INVALID, "Hq must be a positive multiple of Hkv");
  if ((long)B * Hq * ((n_s + 31) / 32) > INT_MAX / 2 || (long)m * dh > INT_MAX / 2 ||
      (long)n_s * dh > INT_MAX / 2)
    return fail(BC_E_CAPACITY, "attention problem too large");
  bc::AttnArgs a{};
  a.q = q;
  a.q_sb = (long)Hq * n_s * dh;
  a.q_sh = (long)n_s * dh;
  a.q_sr = dh;
  a.kp = k_pre;
  a.vp = v_pre;
  a.p_sb = m > 0 ? pre_sb : 0;
  a.p_sh = (long)m * dh;
  a.ks = k_suf;
  a.vs = v_suf;
  a.s_sb = (long)Hkv * n_s * dh;
  a.s_sh = (long)n_s * dh;
  a.s_sr = dh;
  a.out = out;
  a.o_sb = (long)Hq * n_s * dh;
  a.o_sh = (long)n_s * dh;
  a.o_sr = dh;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.m = m;
  a.n_s = n_s;
  a.dh = dh;
  a.scale = scale;
  a.out_f32 = 1;
  BC_HIP(bc::attention(a, (hipStream_t)stream));
  return ok();
}


struct ProfilePlan {
  size_t step = 0, store = 0, out = 0, partial = 0, total = 0;
};

bc::CosView kv_view(const bc_model_config& c, int m, int B) {
  bc::CosView v{};
  v.L = c.n_layers;
  v.P = 2;
  v.H = c.n_kv_heads;
  v.E = (long)m * c.head_dim;
  v.B = B;
  return v;
}

ProfilePlan profile_plan(const bc_model* model, int m, int B, int n_s) {
  ProfilePlan pp;
  const bc_model_config& c = model->cfg;
  Bump b;
  const size_t ws = bc_step_workspace_bytes(model, m, B, n_s, 0);
  if (!ws) return pp;
  pp.step = b.take(ws);
  pp.store = b.take(deep_layout(c, m, B, n_s, 0).total);
  pp.out = b.take((size_t)B * n_s * c.hidden * 4);
  pp.partial = b.take(bc::kv_cosine_partial_bytes(kv_view(c, m, B)));
  pp.total = b.at;
  return pp;
}

}  // namespace

extern "C" {

const char* bc_last_error(void) { return g_err; }

bc_status bc_model_create(const bc_model_config* cfg, const bc_layer_weights* layers,
                          int cache_capacity, bc_model** out) try {
  if (!cfg || !layers || !out) return fail(BC_E_INVALID, "null argument");
  std::string why;
  if (!config_ok(*cfg, &why)) return fail(BC_E_INVALID, "%s", why.c_str());
  if (cache_capacity < 1) return fail(BC_E_INVALID, "cache_capacity must be >= 1");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const bc_layer_weights& w = layers[l];
    if (!w.w_qkv || !w.w_o || !w.w_gate_up || !w.w_down || !w.attn_norm || !w.ffn_norm)
      return fail(BC_E_INVALID, "layer %d has a null weight pointer", l);
    if (misaligned(w.w_qkv) || misaligned(w.w_o) || misaligned(w.w_gate_up) || misaligned(w.w_down) ||
        misaligned(w.attn_norm) || misaligned(w.ffn_norm) || misaligned(w.b_qkv))
      return fail(BC_E_INVALID, "layer %d has a weight pointer that is not 16-byte aligned", l);
  }
  bc_model* m = new (std::nothrow) bc_model(*cfg, layers, cache_capacity);
  if (!m) return fail(BC_E_OOM, "host allocation of the model failed");
  try {
    std::lock_guard<std::mutex> lk(g_models_mu);
    g_models.insert(m);
  } catch (...) {
    delete m;
    throw;
  }
  *out = m;
  return ok();
} catch (...) {
  return host_exception();
}

bc_status bc_model_destroy(bc_model* model) try {
  {
    std::lock_guard<std::mutex> lk(g_models_mu);
    if (!model || g_models.erase(model) == 0) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  }
  delete model;
  return ok();
} catch (...) {
  return host_exception();
}

size_t bc_prefix_cache_bytes(const bc_model* model, int m, int n_layers_to_cache) try {
  if (!live(model) || m < 1 || n_layers_to_cache < 0 || n_layers_to_cache > model->cfg.n_layers) return 0;
  return entry_layout(model->cfg, m, n_layers_to_cache).total;
} catch (...) {
  return 0;
}

size_t bc_cache_offset(const bc_model* model, int m, int Lc, int layer, int part, int head,
                       int pos, int dim) try {
  const size_t bad = (size_t)-1;
  if (!live(model) || m < 1 || Lc < 0 || Lc > model->cfg.n_layers) return bad;
  const bc_model_config& c = model->cfg;
  const EntryLayout e = entry_layout(c, m, Lc);
  if (pos < 0 || pos >= m || dim < 0) return bad;
  if (part == 0 || part == 1) {
    if (layer < 0 || layer >= Lc || head < 0 || head >= c.n_kv_heads || dim >= c.head_dim) return bad;
    return ((size_t)(layer * 2 + part)) * e.kv_layer +
           (((size_t)head * m + pos) * c.head_dim + dim) * 2;
  }
  if (part == 2) {
    if (layer < 0 || layer >= e.n_h || dim >= c.hidden) return bad;
    return e.h_off + (size_t)layer * e.h_layer + ((size_t)pos * c.hidden + dim) * 4;
  }
  return bad;
} catch (...) {
  return 0;
}

size_t bc_populate_workspace_bytes(const bc_model* model, int m) try {
  if (!live(model) || m < 1) return 0;
  return make_plan(model->cfg, m, m, false, m).total;
} catch (...) {
  return 0;
}

bc_status bc_prefix_populate(bc_model* model, uint64_t key, const void* x_prefix, int m,
                             int n_layers_to_cache, void* cache_mem, size_t cache_bytes,
                             void* workspace, size_t ws_bytes, void* stream,
                             uint64_t* evicted_key, int* evicted) try {
  if (evicted) *evicted = 0;
  if (evicted_key) *evicted_key = 0;
  if (!live(model) || !x_prefix || !cache_mem || !workspace) return fail(BC_E_INVALID, "null argument");
  if (misaligned(x_prefix)) return fail(BC_E_INVALID, "x_prefix must be 16-byte aligned");
  const bc_model_config& c = model->cfg;
  const int Lc = n_layers_to_cache;
  if (m < 1) return fail(BC_E_INVALID, "prefix length m=%d must be >= 1", m);
  if (Lc < 0 || Lc > c.n_layers) return fail(BC_E_INVALID, "n_layers_to_cache=%d outside [0, %d]", Lc, c.n_layers);
  std::string why;
  if (!step_shape_ok(c, m, 1, 1, 0, &why)) return fail(BC_E_INVALID, "%s", why.c_str());
  const EntryLayout e = entry_layout(c, m, Lc);
  if (cache_bytes < e.total) return fail(BC_E_INVALID, "cache_bytes %zu < required %zu", cache_bytes, e.total);
  if ((uintptr_t)cache_mem % kAlign) return fail(BC_E_INVALID, "cache_mem must be 256-byte aligned");
  const Plan p = make_plan(c, m, m, false, m);
  if (ws_bytes < p.total) return fail(BC_E_INVALID, "workspace %zu < required %zu", ws_bytes, p.total);
  if ((uintptr_t)workspace % kAlign) return fail(BC_E_INVALID, "workspace must be 256-byte aligned");
  if (model->table.contains(key)) return fail(BC_E_STATE, "key %016llx is already cached", (unsigned long long)key);

  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  char* cm = (char*)cache_mem;
  float* R = (float*)(ws + p.R);
  const long mh = (long)m * c.hidden;
  BC_LAUNCH(model, BC_K_OTHER, s,
            bc::rope_table((float*)(ws + p.cos), (float*)(ws + p.sin), m, c.head_dim, c.rope_theta, s));
  BC_LAUNCH(model, BC_K_OTHER, s, bc::bf16_to_f32(x_prefix, R, mh, s));
  for (int l = 0; l < Lc || l < e.n_h; ++l) {
    if (l < e.n_h)  // H$[l]: residual entering layer l of the prefix-only forward
      BC_HIP(hipMemcpyAsync(cm + e.h_off + (size_t)l * e.h_layer, R, e.h_layer, hipMemcpyDeviceToDevice, s));
    if (l >= Lc) break;
    char* k_dst = cm + (size_t)(2 * l) * e.kv_layer;
    char* v_dst = cm + (size_t)(2 * l + 1) * e.kv_layer;
    const Seg sg{0, 1, m, 0, nullptr, nullptr, 0, k_dst, v_dst, 0, (long)m * c.head_dim};
    LayerCall lc{R, m, &sg, 1};
    // when no H$ slot keeps the residual this layer produces (Lc = L: the last
    // layer), only its K/V are cached and nothing after Q/K/V is computed
    bc_status st = run_layer(model, l, lc, ws, p, s, l + 1 >= e.n_h ? LayerPart::kKvOnly : LayerPart::kAll);
    if (st != BC_OK) return st;
  }
  bc::CacheEntry ce;
  ce.m = m;
  ce.n_layers = Lc;
  ce.mem = cache_mem;
  ce.bytes = cache_bytes;
  uint64_t ev = 0;
  const bool did = model->table.insert(key, ce, &ev);
  if (did) {
    if (evicted) *evicted = 1;
    if (evicted_key) *evicted_key = ev;
  }
  return ok();
} catch (...) {
  return host_exception();
}

bc_status bc_prefix_lookup(const bc_model* model, uint64_t key, int* m_out, int* n_layers_out) try {
  if (!live(model)) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  const bc::CacheEntry* e = model->table.find(key);
  if (!e) return fail(BC_E_NOT_FOUND, "key %016llx is not cached", (unsigned long long)key);
  if (m_out) *m_out = e->m;
  if (n_layers_out) *n_layers_out = e->n_layers;
  return ok();
} catch (...) {
  return host_exception();
}

bc_status bc_prefix_invalidate(bc_model* model, uint64_t key) try {
  if (!live(model)) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  if (!model->table.erase(key)) return fail(BC_E_NOT_FOUND, "key %016llx is not cached", (unsigned long long)key);
  return ok();
} catch (...) {
  return host_exception();
}

bc_status bc_cache_keys(const bc_model* model, uint64_t* keys, int max_keys, int* n_out) try {
  if (!live(model) || !n_out || max_keys < 0 || (max_keys > 0 && !keys)) return fail(BC_E_INVALID, "bad argument");
  int i = 0;
  for (uint64_t k : model->table.order()) {
    if (i < max_keys) keys[i] = k;
    ++i;
  }
  *n_out = i;
  return ok();
} catch (...) {
  return host_exception();
}

uint64_t bc_prefix_key(const int32_t* token_ids, size_t n) try {
  // little-endian int32 bytes, independent of the host's byte order
  std::vector<unsigned char> bytes(n * 4);
  for (size_t i = 0; i < n; ++i) {
    const uint32_t v = (uint32_t)token_ids[i];
    for (int b = 0; b < 4; ++b) bytes[i * 4 + b] = (unsigned char)(v >> (8 * b));
  }
  return bc::xxh64(bytes.data(), bytes.size(), 0);
} catch (...) {
  return 0;
}

size_t bc_step_workspace_bytes(const bc_model* model, int m, int B, int n_s, int d) try {
  if (!live(model)) return 0;
  return step_workspace(model, &m, &B, 1, n_s, d);
} catch (...) {
  return 0;
}

size_t bc_step_multi_workspace_bytes(const bc_model* model, const uint64_t* keys, const int* counts,
                                     int n_groups, int n_s, int d) try {
  if (!live(model) || !keys || !counts || n_groups < 1 || n_groups > kMaxGroups) return 0;
  std::vector<int> ms(n_groups);
  for (int g = 0; g < n_groups; ++g) {
    const bc::CacheEntry* e = model->table.find(keys[g]);
    if (!e) return 0;
    ms[g] = e->m;
  }
  return step_workspace(model, ms.data(), counts, n_groups, n_s, d);
} catch (...) {
  return 0;
}

bc_status bc_step_plan(const bc_model* model, int m, int B, int n_s, int d, int* rows,
                       int* pos_base, int* reads_kv, int* reads_h) try {
  if (!live(model)) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  std::string why;
  if (!step_shape_ok(model->cfg, m, B, n_s, d, &why)) return fail(BC_E_INVALID, "%s", why.c_str());
  const int L = model->cfg.n_layers;
  for (int l = 0; l < L; ++l) {
    const bool shallow = l < d;
    if (rows) rows[l] = shallow ? B * n_s : B * (m + n_s);
    if (pos_base) pos_base[l] = shallow ? m : 0;
    if (reads_kv) reads_kv[l] = shallow ? 1 : 0;
  }
  if (reads_h) *reads_h = d < L ? d : -1;
  return ok();
} catch (...) {
  return host_exception();
}


bc_status bc_step_forward(bc_model* model, uint64_t key, const void* x_suffix, int B, int n_s,
                          int d, float* out, void* workspace, size_t ws_bytes, void* stream) try {
  const Group g{key, B};
  return step_impl(model, &g, 1, x_suffix, n_s, d, BC_DEEP_REFRESH, nullptr, 0, out, workspace,
                   ws_bytes, stream);
} catch (...) {
  return host_exception();
}

size_t bc_deep_store_bytes(const bc_model* model, int m, int B, int n_s, int d) try {
  if (!live(model)) return 0;
  std::string why;
  if (!step_shape_ok(model->cfg, m, B, n_s, d, &why)) return 0;
  return deep_layout(model->cfg, m, B, n_s, d).total;
} catch (...) {
  return 0;
}

size_t bc_deep_store_offset(const bc_model* model, int m, int B, int n_s, int d, int layer,
                            int part, int req, int head, int pos, int dim) try {
  const size_t bad = (size_t)-1;
  if (!live(model)) return bad;
  const bc_model_config& c = model->cfg;
  std::string why;
  if (!step_shape_ok(c, m, B, n_s, d, &why)) return bad;
  if (layer < d || layer >= c.n_layers || part < 0 || part > 1 || req < 0 || req >= B ||
      head < 0 || head >= c.n_kv_heads || pos < 0 || pos >= m + n_s || dim < 0 || dim >= c.head_dim)
    return bad;
  const DeepLayout dl = deep_layout(c, m, B, n_s, d);
  return (size_t)(2 * (layer - d) + part) * dl.part +
         ((size_t)req * dl.sb + (size_t)head * dl.sh + (size_t)pos * c.head_dim + dim) * 2;
} catch (...) {
  return 0;
}

bc_status bc_deep_store_reset(bc_model* model, const void* deep_store) try {
  if (!live(model)) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  model->deep_tags.erase((uintptr_t)deep_store);
  return ok();
} catch (...) {
  return host_exception();
}

int bc_is_refresh_step(int t, int delta) try {
  if (t < 1 || delta < 1) return -1;
  return (t - 1) % delta == 0 ? 1 : 0;
} catch (...) {
  return -1;
}

bc_status bc_step_forward_deep(bc_model* model, uint64_t key, const void* x_suffix, int B,
                               int n_s, int d, int mode, void* deep_store, size_t store_bytes,
                               float* out, void* workspace, size_t ws_bytes, void* stream) try {
  const Group g{key, B};
  return step_impl(model, &g, 1, x_suffix, n_s, d, mode, deep_store, store_bytes, out, workspace,
                   ws_bytes, stream);
} catch (...) {
  return host_exception();
}

bc_status bc_step_forward_multi(bc_model* model, const uint64_t* keys, const int* counts,
                                int n_groups, const void* x_suffix, int n_s, int d, float* out,
                                void* workspace, size_t ws_bytes, void* stream) try {
  if (!keys || !counts) return fail(BC_E_INVALID, "null argument");
  if (n_groups < 1 || n_groups > kMaxGroups)
    return fail(BC_E_INVALID, "n_groups=%d outside [1, %d]", n_groups, kMaxGroups);
  std::vector<Group> gs(n_groups);
  for (int g = 0; g < n_groups; ++g) gs[g] = Group{keys[g], counts[g]};
  return step_impl(model, gs.data(), n_groups, x_suffix, n_s, d, BC_DEEP_REFRESH, nullptr, 0, out,
                   workspace, ws_bytes, stream);
} catch (...) {
  return host_exception();
}

// ------------------------------------------------------- shared-prefix profiling


size_t bc_profile_workspace_bytes(const bc_model* model, int m, int B, int n_s) try {
  if (!live(model)) return 0;
  return profile_plan(model, m, B, n_s).total;
} catch (...) {
  return 0;
}

bc_status bc_profile_similarity(bc_model* model, uint64_t key, const void* x_suffix, int B, int n_s,
                                double* sims, void* workspace, size_t ws_bytes, void* stream) try {
  if (!live(model) || !x_suffix || !sims || !workspace) return fail(BC_E_INVALID, "null argument");
  if (misaligned(x_suffix) || misaligned(sims)) return fail(BC_E_INVALID, "x_suffix and sims must be 16-byte aligned");
  const bc::CacheEntry* ent = model->table.find(key);
  if (!ent) return fail(BC_E_NOT_FOUND, "key %016llx is not cached", (unsigned long long)key);
  const bc_model_config& c = model->cfg;
  const int L = c.n_layers, m = ent->m;
  if (ent->n_layers != L)
    return fail(BC_E_INVALID, "profiling needs KV$ of all %d layers; the entry caches %d", L, ent->n_layers);
  std::string why;
  if (!step_shape_ok(c, m, B, n_s, 0, &why)) return fail(BC_E_INVALID, "%s", why.c_str());
  if ((long)L * 2 * c.n_kv_heads > 65535)
    return fail(BC_E_CAPACITY, "similarity reduction supports at most 65535 (layer, K/V, head) blocks");
  const ProfilePlan pp = profile_plan(model, m, B, n_s);
  if (!pp.total) return fail(BC_E_INVALID, "invalid profiling shape");
  if (ws_bytes < pp.total) return fail(BC_E_INVALID, "workspace %zu < required %zu", ws_bytes, pp.total);
  if ((uintptr_t)workspace % kAlign) return fail(BC_E_INVALID, "workspace must be 256-byte aligned");
  char* ws = (char*)workspace;
  hipStream_t s = (hipStream_t)stream;
  // KV^ref_{l,1}: the un-cached forward of (p, z) at the first step (d = 0),
  // every layer's K/V of every row written to the deep store
  const Group g{key, B};
  bc_status st = step_impl(model, &g, 1, x_suffix, n_s, 0, BC_DEEP_REFRESH, ws + pp.store,
                           pp.out - pp.store, (float*)(ws + pp.out), ws + pp.step, pp.store - pp.step,
                           stream);
  model->deep_tags.erase((uintptr_t)(ws + pp.store));
  if (st != BC_OK) return st;
  const EntryLayout e = entry_layout(c, m, L);
  const DeepLayout dl = deep_layout(c, m, B, n_s, 0);
  const char* cm = (const char*)ent->mem;
  // every layer in one reduction: layer l's KV$ (K then V, [Hkv][m][dh] each)
  // against each request's prefix rows of layer l in the store
  bc::CosView v = kv_view(c, m, B);
  v.a = cm;
  v.a_layer = (long)e.kv_layer;   // elements: 2 blocks of kv_layer bytes
  v.a_part = (long)(e.kv_layer / 2);
  v.a_head = (long)m * c.head_dim;
  v.r = ws + pp.store;
  v.r_layer = (long)dl.part;
  v.r_part = (long)(dl.part / 2);
  v.r_req = dl.sb;
  v.r_head = dl.sh;
  BC_LAUNCH(model, BC_K_KVSIM, s, bc::kv_cosine(v, (double*)(ws + pp.partial), sims, L, 1, s));
  return ok();
} catch (...) {
  return host_exception();
}

size_t bc_cosine_workspace_bytes(long n) try {
  if (n <= 0 || n % 8) return 0;
  bc::CosView v{};
  v.L = v.P = v.H = v.B = 1;
  v.E = n;
  return bc::kv_cosine_partial_bytes(v);
} catch (...) {
  return 0;
}

bc_status bc_cosine_similarity(const void* a, const void* b, long n, double* out, void* workspace,
                               size_t ws_bytes, void* stream) try {
  if (!a || !b || !out || !workspace) return fail(BC_E_INVALID, "null argument");
  if (n <= 0 || n % 8) return fail(BC_E_INVALID, "n=%ld must be a positive multiple of 8", n);
  if (misaligned(a) || misaligned(b) || misaligned(out)) return fail(BC_E_INVALID, "a, b and out must be 16-byte aligned");
  const size_t need = bc_cosine_workspace_bytes(n);
  if (ws_bytes < need) return fail(BC_E_INVALID, "workspace %zu < required %zu", ws_bytes, need);
  bc::CosView v{};
  v.a = a;
  v.r = b;
  v.L = v.P = v.H = v.B = 1;
  v.E = n;
  BC_HIP(bc::kv_cosine(v, (double*)workspace, out, 1, 1, (hipStream_t)stream));
  return ok();
} catch (...) {
  return host_exception();
}

bc_status bc_cosine_similarity_noalloc(const void* a, const void* b, long n, double* out,
                                       void* stream) try {
  if (!a || !b || !out) return fail(BC_E_INVALID, "null argument");
  if (n <= 0 || n % 8) return fail(BC_E_INVALID, "n=%ld must be a positive multiple of 8", n);
  if (misaligned(a) || misaligned(b) || misaligned(out)) return fail(BC_E_INVALID, "a, b and out must be 16-byte aligned");
  const size_t need = bc_cosine_workspace_bytes(n);
  if (need > bc::cosine_scratch_bytes())
    return fail(BC_E_CAPACITY, "n=%ld exceeds the %ld elements the static scratch (%zu bytes) serves",
                n, bc::cosine_scratch_max_elements(), bc::cosine_scratch_bytes());
  double* scr = nullptr;
  BC_HIP(bc::cosine_scratch(&scr));
  bc::CosView v{};
  v.a = a;
  v.r = b;
  v.L = v.P = v.H = v.B = 1;
  v.E = n;
  BC_HIP(bc::kv_cosine(v, scr, out, 1, 1, (hipStream_t)stream));
  return ok();
} catch (...) {
  return host_exception();
}

int bc_shallow_depth(const double* sims, int n_layers, double tau) try {
  if (!sims || n_layers < 0) return -1;
  int b = 0;
  while (b < n_layers && sims[b] >= tau) ++b;
  return b;
} catch (...) {
  return -1;
}

bc_status bc_build_depth_table(const double* ratios, const int* depths, int n, int n_buckets,
                               int* table) try {
  if (!ratios || !depths || !table || n < 0 || n_buckets < 1) return fail(BC_E_INVALID, "bad argument");
  std::vector<long> sum(n_buckets + 1, 0), cnt(n_buckets + 1, 0);
  for (int i = 0; i < n; ++i) {
    const double k = ratios[i] * n_buckets;
    const long kr = lround(k);
    if (kr < 1 || kr > n_buckets || fabs((double)kr / n_buckets - ratios[i]) >= 1e-9)
      return fail(BC_E_INVALID, "ratio %g of request %d is not a bucket value k/%d", ratios[i], i, n_buckets);
    if (depths[i] < 0) return fail(BC_E_INVALID, "depth %d of request %d is negative", depths[i], i);
    sum[kr] += depths[i];
    cnt[kr] += 1;
  }
  table[0] = -1;
  for (int k = 1; k <= n_buckets; ++k) table[k] = cnt[k] ? (int)(sum[k] / cnt[k]) : -1;
  return ok();
} catch (...) {
  return host_exception();
}

int bc_depth_lookup(const int* table, int n_buckets, double r) try {
  if (!table || n_buckets < 1 || !(r >= 0.0)) return -1;
  long k = (long)floor(r * n_buckets + 1e-9);
  if (k > n_buckets) k = n_buckets;
  for (; k >= 1; --k)
    if (table[k] >= 0) return table[k];
  return 0;
} catch (...) {
  return -1;
}

bc_status bc_profile_begin(bc_model* model, unsigned kernel_mask) try {
  if (!live(model)) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  model->prof.mask = kernel_mask;
  model->prof.used = 0;
  model->prof.recs.clear();
  return ok();
} catch (...) {
  return host_exception();
}

bc_status bc_profile_end(bc_model* model, double* ms, int* launches) try {
  if (!live(model)) return fail(BC_E_INVALID, "null, unknown or destroyed model");
  Profiler& p = model->prof;
  p.mask = 0;
  double acc[BC_K_COUNT] = {0};
  int cnt[BC_K_COUNT] = {0};
  if (p.used) BC_HIP(hipEventSynchronize(p.pool[p.used - 1]));
  for (const Profiler::Rec& r : p.recs) {
    float t = 0.f;
    BC_HIP(hipEventElapsedTime(&t, p.pool[r.start], p.pool[r.stop]));
    acc[r.kind] += t;
    cnt[r.kind] += 1;
  }
  p.recs.clear();
  p.used = 0;
  for (int k = 0; k < BC_K_COUNT; ++k) {
    if (ms) ms[k] = acc[k];
    if (launches) launches[k] = cnt[k];
  }
  return ok();
} catch (...) {
  return host_exception();
}


bc_status bc_shared_prefix_attention(const void* q, const void* k_pre, const void* v_pre,
                                     const void* k_suf, const void* v_suf, float* out, int B,
                                     int Hq, int Hkv, int m, int n_s, int dh, float scale,
                                     void* stream) try {
  return prefix_attention(q, k_pre, v_pre, 0, k_suf, v_suf, out, B, Hq, Hkv, m, n_s, dh, scale,
                          stream);
} catch (...) {
  return host_exception();
}

bc_status bc_request_prefix_attention(const void* q, const void* k_pre, const void* v_pre,
                                      const void* k_suf, const void* v_suf, float* out, int B,
                                      int Hq, int Hkv, int m, int n_s, int dh, float scale,
                                      void* stream) try {
  return prefix_attention(q, k_pre, v_pre, (long)Hkv * m * dh, k_suf, v_suf, out, B, Hq, Hkv, m,
                          n_s, dh, scale, stream);
} catch (...) {
  return host_exception();
}

}  // extern "C"
