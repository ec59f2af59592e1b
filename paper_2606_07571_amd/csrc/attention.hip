// Shared-prefix bidirectional attention on gfx950 (Eq. 2 over [prefix ; own
// suffix], the shallow-layer form of Eq. 4).  With m = 0 the same kernel is
// the deep layers' full attention of every request over its own sequence, and
// with a per-request prefix (p_sb != 0) it is the deep layers' attention of a
// step that reuses each request's own prefix K/V (second case of Eq. 5).
//
// Work decomposition.  For one KV head g, the query rows of every request b
// and every query head of g's group are cut into chunks of 32 rows
// (b, head, i0); a workgroup of 8 waves takes 8 consecutive chunks, one per
// wave.  The key sequence the workgroup walks is
//     [the prefix tiles of g]  then, for each distinct request among its
//     chunks, [that request's suffix tiles of g],
// in tiles of 64 keys staged through LDS.  A prefix tile is loaded once per
// workgroup and consumed by all 8 waves, whatever request or query head they
// serve: one LDS copy of the shared prefix feeds the workgroup's 256 query
// rows.  Those rows span several requests only when a request brings fewer
// than 8 chunks per KV head (GQA group size x suffix chunks < 8, e.g. two
// 64-row suffixes); at the large shapes (suffix 256-512 rows) a workgroup
// serves one request, and the prefix tiles shared by the requests are reused
// from L2 and the last-level cache, not from LDS.  Putting several requests
// into one workgroup there would make every wave walk the other requests'
// suffix tiles masked (2.4x the tiles at the LLaDA-8B shape).  A suffix tile
// is consumed only by the waves of its request.  When every request has its own prefix, the prefix tiles join the
// request's part of the walk: [its prefix tiles ; its suffix tiles].
//
// Per wave the scores are computed transposed, S^T = K . Q^T with
// v_mfma_f32_32x32x16_bf16: a lane then holds 16 scores of ONE query row
// (row l%32, keys 8j + 4*(l/32) + i), so the online-softmax row max needs a
// single cross-lane exchange (lanes l and l^32) per tile and the row sum needs
// none until the end.  The output is accumulated transposed as well,
// O^T += V^T . P^T: the P^T operand comes straight from the score registers
// (no data movement; the MFMA's k order is chosen to match the keys a lane
// already holds) and the V^T operand is read from the row-major V tile with
// transposing LDS reads (ds_read_b64_tr_b16).
// Softmax runs in fp32 in the log2 domain (exp2 with log2(e) folded into the
// scale); P is rounded to bf16 for the P.V product, and the row sums are taken
// on the matrix pipe from the same bf16 probabilities (one 16x16x32 MFMA per
// 16 keys against a 0/1 selector), so the weights that multiply V are the
// ones that are normalised and no vector adds are spent on the sums.
//
// Software pipeline.  Every wave overlaps its own matrix and vector work: in
// step u it runs
//   block A: O^T += V(u-1)^T . P(u-1)^T (16 MFMAs) alongside the softmax of
//            S(u) (P(u) = exp2(...) against the running max, row sums)
//   block B: S(u+1)^T = K(u+1) . Q^T (16 MFMAs) alongside this thread's share
//            of the LDS fill of tile u+2 and the global fetch of tile u+4
// and one barrier.  The MFMAs of a block do not depend on its vector work, so
// the two streams issue side by side, and with two such waves per SIMD the
// vector instructions issue at the SIMD's full rate (one wave alone issues
// one only every other slot).  The online softmax stays exact with a running
// max that moves rarely: the first tile sets it to the tile's row max; after
// that P(u) is formed against it directly and the tile's row sums, which come
// from the matrix pipe anyway, bound every probability.  Only a sum above
// 2^16 (a score far above the running max, or a row that had no valid key
// yet) moves the max to the tile's and forms P(u) again; O, which holds
// P(u-1).V(u-1) computed with the old max once block A is done, is then
// rescaled between the blocks.  Any running max gives the same result up to
// the bf16 rounding of P, since O and the row sum carry the same factor; the
// bound keeps probabilities, and so O and the row sums, far from overflow.
// No row max is taken on the common path.
//
// LDS.  Tiles live in a 4-deep ring (tile t in slot t % 4): step u reads
// V(u-1) and K(u+1) and fills tile u+2, whose slot last held tile u-2.  The
// global fetch of a tile lands in one of two register staging sets (tile t in
// set t % 2) two steps before its LDS fill, so a fetch that misses the L2 has
// two steps to arrive.
// K and V tiles are both stored as they are in memory, one key per row, filled
// with 16-byte writes.  K rows are padded by 16 bytes (dh+8 elements), so the
// 16 rows that one K fragment read touches fall into distinct bank groups; V
// rows by 64 bytes (dh+32), so the 4 rows x 32 bytes of each 16-lane group of
// a transposing read, and both groups of a half wave, hit distinct banks.
// Every fragment of a tile sits at a compile-time offset from one per-lane
// base.  A V^T fragment (8 keys of one dim per lane) is two transposing reads:
// keys 16s + 4h + {0..3} and 16s + 8 + 4h + {0..3} for lane half h, the order
// of the P^T operand's k slots.  (An earlier V^T copy transposed in registers
// before the fill measured the same on the large shapes and 2-8% slower on
// short walks.)
// Global fetches are buffer loads whose descriptor covers exactly the tile's
// valid rows, so key rows past the end of a partial tile (and whole tiles past
// the end of the sequence) read as zero with no masking code.  Key rows of
// every K/V operand are dh elements apart.
#include "device_common.hpp"
#include "kernels.hpp"

#include <type_traits>

namespace bc {
namespace {

constexpr int KT = 64;  // keys per LDS tile

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

template <int DH, bool OUT_F32>
__global__ void __launch_bounds__(512) attn_il_kernel(AttnArgs a, int CQ, int wg_per_group) {
  constexpr int NW = 8, QR = 32;
  constexpr int KCH = DH / 8;                  // 16-byte chunks per key row
  constexpr int KROW = DH + 8;                 // K row stride in LDS (elements)
  constexpr int VROW = DH + 32;                // V row stride in LDS (elements): rows 16 banks apart
  constexpr int KTILE = KT * KROW, VTILE = KT * VROW, SLOT = KTILE + VTILE;
  constexpr int NBUF = 4;
  constexpr int K_PER = KT * KCH / 512;        // 16-byte K chunks per thread per tile
  constexpr int NB = DH / 32, NKK = DH / 16, NS = KT / 16;
  constexpr int RSRC_W3 = 0x00020000;          // raw buffer, 32-bit dwords (gfx9 family)

  __shared__ __attribute__((aligned(16))) bf16 smem[NBUF * SLOT];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, c = lane & 31;

  const int lid = xcd_remap(blockIdx.x, gridDim.x);
  const int g = lid / wg_per_group, wgi = lid % wg_per_group;
  const int G = a.Hq / a.Hkv;
  const int per_req = G * CQ;
  const int total = a.B * per_req;
  const int c0 = wgi * NW;
  const int c_last = min(c0 + NW, total) - 1;
  const int b_lo = c0 / per_req, b_hi = c_last / per_req;

  const int my = c0 + wave;
  const bool active = my < total;
  const int cc = active ? my : c_last;
  const int b = cc / per_req;
  const int rem = cc - b * per_req;
  const int hq = g * G + rem / CQ;
  const int i0 = (rem % CQ) * QR;
  const int qrow = i0 + c;
  const bool row_ok = active && qrow < a.n_s;

  bf16x8 qf[NKK];
  {
    const bf16* qp = (const bf16*)a.q + b * a.q_sb + hq * a.q_sh + (long)(row_ok ? qrow : 0) * a.q_sr;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok) v = *reinterpret_cast<const u32x4*>(qp + kk * 16 + half * 8);
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  // Tile walk: the shared prefix (when one copy serves all requests), then
  // for each distinct request of the workgroup its own prefix (when every
  // request has one) and its suffix.  The walk is a cursor over these
  // segments: the fetch of a tile reads the cursor and advances it by one
  // tile, a few scalar operations, with a segment change only at segment
  // ends.  Fetches happen in tile order, once per tile.
  const int TP = cdiv(a.m, KT), TS = cdiv(a.n_s, KT);
  const bool own_pre = a.p_sb != 0;
  const int SP = own_pre ? 0 : TP, PR = (own_pre ? TP : 0) + TS;
  const int n_tiles = SP + (b_hi - b_lo + 1) * PR;
  const bf16* const kp0 = (const bf16*)a.kp + g * a.p_sh;
  const bf16* const vp0 = (const bf16*)a.vp + g * a.p_sh;
  const bf16* const ks0 = (const bf16*)a.ks + g * a.s_sh;
  const bf16* const vs0 = (const bf16*)a.vs + g * a.s_sh;
  const bf16* wk = kp0;   // first key row of the next tile to fetch
  const bf16* wv = vp0;
  int w_left = 0;         // key rows from there to the end of its segment
  int w_req = 0;          // request of the segment, -1 for the shared prefix
  int w_phase = 0;        // 0 shared prefix, 1 own prefix, 2 suffix
  // enter segment (phase, req), skipping empty ones; past the last request
  // the walk stays at the end (w_left = 0: empty tiles)
  auto enter = [&](int phase, int req) __attribute__((always_inline)) {
    for (;;) {
      if (req > b_hi) { w_left = 0; w_req = req; w_phase = 2; return; }
      if (phase == 0) {
        if (SP > 0) { wk = kp0; wv = vp0; w_left = a.m; w_req = -1; w_phase = 0; return; }
        phase = own_pre ? 1 : 2;
        req = b_lo;
      } else if (phase == 1) {
        if (a.m > 0) {
          wk = kp0 + req * a.p_sb;
          wv = vp0 + req * a.p_sb;
          w_left = a.m; w_req = req; w_phase = 1;
          return;
        }
        phase = 2;
      } else {
        wk = ks0 + req * a.s_sb;
        wv = vs0 + req * a.s_sb;
        w_left = a.n_s; w_req = req; w_phase = 2;
        return;
      }
    }
  };
  // -1 when the keys of the segment at the cursor are this wave's (the shared
  // prefix, or its own request's), else 0: set once per segment
  int w_mask = 0;
  auto enter_seg = [&](int phase, int req) __attribute__((always_inline)) {
    enter(phase, req);
    w_mask = (active && (w_req < 0 || w_req == b)) ? -1 : 0;
  };
  enter_seg(0, b_lo);
  // valid keys of each fetched tile for this wave (0 for tiles of another
  // request and past the end), queued from fetch to use: tiles u..u+3
  int nvq0 = 0, nvq1 = 0, nvq2 = 0, nvq3 = 0, nvq4 = 0;

  // this thread's share of a fill: K and V chunks q = tid + 512p (row q / KCH,
  // chunk q % KCH)
  int kg_off[K_PER], ks_off[K_PER];
#pragma unroll
  for (int p = 0; p < K_PER; ++p) {
    const int q = tid + 512 * p, r = q / KCH, kc = q % KCH;
    kg_off[p] = (r * DH + kc * 8) * 2;                 // bytes from the tile's first row
    ks_off[p] = r * KROW + kc * 8;                     // elements in the LDS K tile
  }
  int vs_off[K_PER];
#pragma unroll
  for (int p = 0; p < K_PER; ++p) {
    const int q = tid + 512 * p, r = q / KCH, kc = q % KCH;
    vs_off[p] = KTILE + r * VROW + kc * 8;             // elements in the LDS slot
  }

  u32x4 kreg[2][K_PER], vreg[2][K_PER];   // two staging sets: tile t in set t % 2
  // fetch of the tile at the cursor, which then moves on; tiles past the end
  // get an empty descriptor, so their loads return zeros
  auto fetch = [&](auto set_c) __attribute__((always_inline)) {
    constexpr int S = decltype(set_c)::value;
    const int nv = min(KT, w_left);
    const int bytes = nv * DH * 2;
    nvq4 = nv & w_mask;
    const auto rk = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(wk), (short)0, bytes, RSRC_W3);
    const auto rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(wv), (short)0, bytes, RSRC_W3);
    if (w_left > KT) {
      wk += KT * DH;
      wv += KT * DH;
      w_left -= KT;
    } else if (w_req <= b_hi) {
      if (w_phase == 0) enter_seg(own_pre ? 1 : 2, b_lo);
      else if (w_phase == 1) enter_seg(2, w_req);
      else enter_seg(own_pre ? 1 : 2, w_req + 1);
    }
#pragma unroll
    for (int p = 0; p < K_PER; ++p) kreg[S][p] = __builtin_amdgcn_raw_buffer_load_b128(rk, kg_off[p], 0, 0);
#pragma unroll
    for (int p = 0; p < K_PER; ++p) vreg[S][p] = __builtin_amdgcn_raw_buffer_load_b128(rv, kg_off[p], 0, 0);
  };
  auto stash = [&](int slot, auto set_c) __attribute__((always_inline)) {
    constexpr int S = decltype(set_c)::value;
    bf16* base = smem + slot * SLOT;
#pragma unroll
    for (int p = 0; p < K_PER; ++p) *reinterpret_cast<u32x4*>(base + ks_off[p]) = kreg[S][p];
#pragma unroll
    for (int p = 0; p < K_PER; ++p) *reinterpret_cast<u32x4*>(base + vs_off[p]) = vreg[S][p];
  };

  f32x16 o[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) o[nb] = zero16();
  // running row max m (log2 units) and row sum l
  float m_run = -1e30f;
  // Row sums on the matrix pipe: D(16x16) = A . P^T with A rows 0 and 1
  // selecting the lanes that hold query rows c and c + 16 (lanes 0, 32 and
  // 17, 49 supply ones), so lanes 0..15 accumulate the sums of rows l and
  // l + 16 of the bf16 probabilities in elements 0 and 1.
  f32x4 lacc = {0.f, 0.f, 0.f, 0.f};
  bf16x8 ones_sel;
  {
    const uint32_t w1 = (lane == 0 || lane == 32 || lane == 17 || lane == 49) ? 0x3f803f80u : 0u;
    const u32x4 v = {w1, w1, w1, w1};
    ones_sel = __builtin_bit_cast(bf16x8, v);
  }
  const float sl2 = a.scale * 1.4426950408889634f;
  const int k_rd = c * KROW + half * 8;                // lane's K fragment base
  // V^T fragment (dims nb*32 + c, the 8 keys of k slots (half, 0..7) of k
  // step s) from two transposed reads of the row-major V tile: in each group
  // of 16 lanes (G = lane / 16, j = lane % 16) lane j addresses dims
  // 16(G%2) + 4(j%4) .. +3 of key row 4(G/2) + j/4 (+ 16s, + 8 for the keys of
  // slots 4..7), and lane i of the group receives dim i of the 4 rows
  // addressed by lanes 4k + i/4, k = 0..3.
  const int v_rd = KTILE + (4 * (lane >> 5) + ((lane & 15) >> 2)) * VROW + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  auto vfrag = [&](const bf16* vt, int nb, int s) __attribute__((always_inline)) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(vt + 16 * s * VROW + nb * 32));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(vt + (16 * s + 8) * VROW + nb * 32));
    const s16x4 w[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, w);
  };
  auto pv = [&](int t, const bf16x8 (&p)[NS]) __attribute__((always_inline)) {
    const bf16* vt = smem + (t % NBUF) * SLOT + v_rd;
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) o[nb] = mfma_32x32x16(vfrag(vt, nb, s), p[s], o[nb]);
  };
  auto qk = [&](int t, f32x16 (&sc)[2]) __attribute__((always_inline)) {
    const bf16* kt = smem + (t % NBUF) * SLOT + k_rd;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kt + kb * 32 * KROW + kk * 16);
        sc[kb] = mfma_32x32x16(kf, qf[kk], kk == 0 ? zero16() : sc[kb]);
      }
  };
  // scores of a partial tile past its valid keys -> -inf; lane (half, c) holds
  // key 32kb + 8(e/4) + 4half + e%4 of query row c in element e of block kb
  // (branch-free bit select: compares would each hold a scalar mask)
  auto mask = [&](f32x16 (&sc)[2], int nv) __attribute__((always_inline)) {
    const int t = nv - 1 - 4 * half;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = (t - (kb * 32 + 8 * (e >> 2) + (e & 3))) >> 31;   // -1: key >= nv
        sc[kb][e] = __int_as_float((__float_as_int(sc[kb][e]) & ~m) | (int(0xff800000u) & m));
      }
  };
  // P^T operand of k step s: slot (half, e) is key 16s + 8(e/4) + 4half +
  // e%4, i.e. score element 8(s%2) + e of block s/2
  auto probs = [&](const f32x16 (&sc)[2], int s) __attribute__((always_inline)) {
    uint32_t pw[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int e0 = 8 * (s & 1) + 2 * w;
      const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[s >> 1][e0], sl2, -m_run));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[s >> 1][e0 + 1], sl2, -m_run));
      pw[w] = pack_bf16x2(p0, p1);
    }
    const u32x4 pv4 = {pw[0], pw[1], pw[2], pw[3]};
    return __builtin_bit_cast(bf16x8, pv4);
  };
  // Row max of the first tile (step 0): the running max moves when some
  // row's tile max exceeds it by more than 8 (log2 units); returns the factor
  // that moves O and the row sum to the new max (1 when it does not move).
  // m starts at -inf, kept finite so that fully masked tiles give
  // exp2(-inf) = 0 and leave it there.
  bool moved = false;   // wave-uniform: the running max moved in this step
  auto new_max = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[kb][e]);
    mx = half_max(mx) * sl2;
    const bool move = __builtin_amdgcn_ballot_w64(mx > m_run + 8.f) != 0;
    moved = move;
    const float m_new = move ? fmaxf(m_run, mx) : m_run;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    return alpha;
  };

  // One step, as a chain of fenced sub-blocks of (up to) 4 MFMAs each: NS
  // P.V sub-blocks (k step s of P(u-1).V(u-1)) and NKK/2 QK sub-blocks (k
  // steps 2j, 2j+1 of S(u+1)).  Each sub-block first issues the LDS fragment
  // reads of the next one (the last reads the next step's first), then its
  // MFMAs interleaved with its share of the vector work, so fragment reads
  // have a whole sub-block to arrive and a wave never waits on LDS with
  // independent work queued behind the wait.
  //   P.V sub-block s:   softmax of S(u): P(u)'s k step s, written into the
  //                      registers the sub-block's MFMAs have just read, and
  //                      its row sums; after the last, the bound check (and,
  //                      rarely, the max move and P(u) again)
  //   QK sub-blocks:     LDS fill of tile u+2, fetch of tile u+3
  // p holds P(u-1) on entry and P(u) on exit; sc holds S(u) on entry and
  // S(u+1) on exit; fr[0] holds the first sub-block's fragments on entry and
  // the next step's on exit.  Tiles the wave does not own (another request's
  // suffix) are fully masked, so their probabilities are zero and the P.V
  // product adds nothing; every MFMA and vector instruction runs
  // unconditionally.
  constexpr int NQS = NKK / 2;                  // QK sub-blocks
  constexpr int NSUB = NS + NQS;
  static_assert(NSUB % 2 == 0, "fragment double buffer parity");
  auto load_sub = [&](int j, int u, bf16x8 (&f)[4]) __attribute__((always_inline)) {
    if (j < NS) {
      const bf16* vt = smem + ((u + NBUF - 1) % NBUF) * SLOT + v_rd;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) f[nb] = vfrag(vt, nb, j);
    } else {
      const bf16* kt = smem + ((u + 1) % NBUF) * SLOT + k_rd;
      const int kk0 = 2 * (j - NS);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        f[i] = *reinterpret_cast<const bf16x8*>(kt + (i & 1) * 32 * KROW + (kk0 + (i >> 1)) * 16);
    }
  };
  auto step = [&](int u, auto has_pv, auto set_c, bf16x8 (&p)[NS], f32x16 (&sc)[2], bf16x8 (&fr)[2][4])
      __attribute__((always_inline)) {
    constexpr bool PV = decltype(has_pv)::value;
    f32x4 ltile = {0.f, 0.f, 0.f, 0.f};
    const int nv = nvq0;
    if (nv < KT) mask(sc, nv);
    if constexpr (!PV) load_sub(NS, u, fr[NS & 1]);
    float alpha = 1.f;
#pragma unroll
    for (int j = 0; j < NSUB; ++j) {
      if (PV || j >= NS) {
        if (j + 1 < NSUB) load_sub(j + 1, u, fr[(j + 1) & 1]);
        else load_sub(0, u + 1, fr[0]);
      }
      if (j < NS) {
        if constexpr (PV) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) o[nb] = mfma_32x32x16(fr[j & 1][nb], p[j], o[nb]);
        }
        if (!PV && j == 0) alpha = new_max(sc);
        p[j] = probs(sc, j);
        // pin P(u)'s step j here: otherwise the compiler defers the softmax
        // past the QK MFMAs and keeps a second copy of S(u) alive
        asm volatile("" : "+v"(p[j]));
        ltile = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones_sel, p[j], ltile, 0, 0, 0);
      } else {
        const int kk0 = 2 * (j - NS);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kk = kk0 + (i >> 1), kb = i & 1;
          sc[kb] = mfma_32x32x16(fr[j & 1][i], qf[kk], kk == 0 ? zero16() : sc[kb]);
        }
        if (j == NS) stash((u + 2) % NBUF, set_c);              // tile u+2, fetched two steps ago
        if (j == NS + 1 || (NQS == 1 && j == NS)) fetch(set_c);   // tile u+4
      }
      // reads first, then MFMAs each followed by a share of the VALU work
      if (PV || j >= NS) {
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
        }
        if (j < NS) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (j == NS - 1) {
        if constexpr (PV) {
          // a row sum above 2^16 (or not finite) means a probability may be:
          // move the max to the tile's and form P(u) and its sums again
          const bool big = __builtin_amdgcn_ballot_w64(!(ltile[0] <= 65536.f && ltile[1] <= 65536.f)) != 0;
          moved = big;
          if (big) {
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
              for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[kb][e]);
            const float m_new = fmaxf(m_run, half_max(mx) * sl2);
            alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            ltile = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < NS; ++s) {
              p[s] = probs(sc, s);
              ltile = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones_sel, p[s], ltile, 0, 0, 0);
            }
          }
        }
        if (moved) {
          // rare: the running max moved; O already holds P(u-1).V(u-1)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[nb][e] *= alpha;
          lacc[0] *= alpha;
          lacc[1] *= __shfl(alpha, (lane & 15) + 16, 64);
        }
        lacc[0] += ltile[0];
        lacc[1] += ltile[1];
      }
    }
    // keep each step's work on its own side of the barrier
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    nvq0 = nvq1;
    nvq1 = nvq2;
    nvq2 = nvq3;
    nvq3 = nvq4;
  };
  using T_ = std::true_type;
  using F_ = std::false_type;

  // prologue: tiles 0 and 1 in LDS, tile 2 in flight, S(0) computed
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  fetch(S0{});
  nvq0 = nvq4;
  fetch(S1{});
  nvq1 = nvq4;
  stash(0, S0{});
  stash(1, S1{});
  fetch(S0{});
  nvq2 = nvq4;
  fetch(S1{});
  nvq3 = nvq4;
  __syncthreads();
  bf16x8 p[NS];
  f32x16 sc[2];
  bf16x8 fr[2][4];
  qk(0, sc);
  // (the last step's S(n_tiles) reads a zero-filled slot and is discarded)
  step(0, F_{}, S0{}, p, sc, fr);
  int u = 1;
  for (; u + 1 < n_tiles; u += 2) {
    step(u, T_{}, S1{}, p, sc, fr);
    step(u + 1, T_{}, S0{}, p, sc, fr);
  }
  if (u < n_tiles) step(u, T_{}, S1{}, p, sc, fr);
  pv(n_tiles - 1, p);

  // Output.  A lane holds dims nb*32 + 8j + 4*half + {0..3} of its query row,
  // so direct stores would write 8 or 16 bytes into each of 32 rows per
  // instruction.  Instead each wave writes its 32 rows into a region of its
  // own in two ring slots no longer in use (every slot but the last tile's,
  // which other waves may still be reading: the final barrier has passed),
  // and reads them back as runs of whole rows (256 bytes of a row per pass
  // of DPP dims at dh = 128, 128 at dh = 64), 16 bytes per lane, so that a
  // store instruction writes 4 (or 8) row runs.  Nothing else touches the
  // region: no barrier.
  const float l0 = __shfl(lacc[0], c & 15, 64), l1 = __shfl(lacc[1], c & 15, 64);
  const float inv = 1.f / (c < 16 ? l0 : l1);
  {
    typedef std::conditional_t<OUT_F32, float, bf16> OT;
    constexpr int ES = sizeof(OT);
    constexpr int RMAX = DH >= 128 ? 256 : 128;          // row bytes per pass at most
    constexpr int DPP = DH * ES > RMAX ? RMAX / ES : DH;  // dims per pass
    constexpr int RBY = DPP * ES;                        // bytes of a row per pass
    constexpr int RST = RBY + 16;                        // LDS row stride (bytes)
    constexpr int LPR = RBY / 16;                        // lanes per row on the way out
    constexpr int RPI = 64 / LPR;                        // rows per store instruction
    static_assert(NW * QR * RST <= 2 * SLOT * 2, "staging must fit in two slots");
    const int busy = (n_tiles - 1) % NBUF;
    const int s0 = busy >= 2 ? 0 : busy + 1;             // first of two free, adjacent slots
    char* reg = reinterpret_cast<char*>(smem + s0 * SLOT) + wave * (QR * RST);
    const int nrow = active ? a.n_s - i0 : 0;            // valid rows of this wave's chunk
    OT* ob = (OT*)a.out + b * a.o_sb + hq * a.o_sh + (long)i0 * a.o_sr;
#pragma unroll
    for (int q = 0; q < DH / DPP; ++q) {
#pragma unroll
      for (int nb = q * DPP / 32; nb < (q + 1) * DPP / 32; ++nb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          char* d = reg + c * RST + (nb * 32 + 8 * j + 4 * half - q * DPP) * ES;
          if constexpr (OUT_F32) {
            const f32x4 v = {o[nb][4 * j] * inv, o[nb][4 * j + 1] * inv, o[nb][4 * j + 2] * inv,
                             o[nb][4 * j + 3] * inv};
            *reinterpret_cast<f32x4*>(d) = v;
          } else {
            const u32x2 v = {pack_bf16x2(o[nb][4 * j] * inv, o[nb][4 * j + 1] * inv),
                             pack_bf16x2(o[nb][4 * j + 2] * inv, o[nb][4 * j + 3] * inv)};
            *reinterpret_cast<u32x2*>(d) = v;
          }
        }
#pragma unroll
      for (int k = 0; k < QR / RPI; ++k) {
        const int row = k * RPI + lane / LPR, ch = lane % LPR;
        const u32x4 v = *reinterpret_cast<const u32x4*>(reg + row * RST + ch * 16);
        if (row < nrow)
          *reinterpret_cast<u32x4*>(ob + (long)row * a.o_sr + q * DPP + ch * (16 / ES)) = v;
      }
    }
  }
}

template <int DH, bool F32>
hipError_t launch_il(const AttnArgs& a, hipStream_t s) {
  if (a.s_sr != DH) return hipErrorInvalidValue;   // key rows must be dh apart
  const int CQ = cdiv(a.n_s, 32);
  const int G = a.Hq / a.Hkv;
  const int wpg = cdiv(a.B * G * CQ, 8);
  const int grid = a.Hkv * wpg;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_il_kernel<DH, F32>), dim3(grid), dim3(512), 0, s, a, CQ, wpg);
  return hipGetLastError();
}

}  // namespace

hipError_t attention(const AttnArgs& a, hipStream_t s) {
  if (a.dh == 128) return a.out_f32 ? launch_il<128, true>(a, s) : launch_il<128, false>(a, s);
  return a.out_f32 ? launch_il<64, true>(a, s) : launch_il<64, false>(a, s);
}

}  // namespace bc
