// Shared-prefix bidirectional attention on gfx950 (Eq. 2 over [prefix ; own
// suffix], the shallow-layer form of Eq. 4).  With m = 0 the same kernel is
// the deep layers' full attention of every request over its own sequence.
//
// Work decomposition.  For one KV head g, the query rows of every request b
// and every query head of g's group are cut into chunks of QB*32 rows
// (b, head, i0); a workgroup of NW waves takes NW consecutive chunks, one per
// wave.  A wave holds QB query blocks of 32 rows, so every K or V fragment it
// reads from LDS feeds QB MFMAs.  The key
// sequence the workgroup walks is
//     [the prefix tiles of g]  then, for each distinct request among its
//     chunks, [that request's suffix tiles of g],
// in tiles of 64 keys staged through LDS.  A prefix tile is loaded once per
// workgroup and consumed by all NW waves, whatever request or query head they
// serve, so one LDS copy of the shared prefix feeds up to NW*32 query rows of
// several requests.  A suffix tile is consumed only by the waves of its
// request.
//
// Per wave the scores are computed transposed, S^T = K . Q^T with
// v_mfma_f32_32x32x16_bf16: a lane then holds 16 scores of ONE query row
// (row l%32, keys 8j + 4*(l/32) + i), so the online-softmax row max needs a
// single cross-lane exchange (lanes l and l^32) per tile and the row sum needs
// none until the end.  The output is accumulated transposed as well,
// O^T += V^T . P^T: the P^T operand comes straight from the score registers
// (no data movement; the MFMA's k order is chosen to match the keys a lane
// already holds) and V^T is read from a transposed LDS copy of the V tile.
// Softmax runs in fp32 in the log2 domain (exp2 with log2(e) folded into the
// scale); P is rounded to bf16 for the P.V product.
#include "device_common.hpp"
#include "kernels.hpp"

namespace bc {
namespace {

constexpr int KT = 64;  // keys per LDS tile

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

// K tile: rows of dh bf16 (KCH 16-byte chunks).  LDS serves 128-bit accesses
// 16 lanes (256 bytes, 64 banks) at a time, and a fragment read touches 16
// consecutive rows at one chunk: with 256-byte rows (dh 128) chunk kc of row r
// is stored at kc ^ (r & 15); with 128-byte rows (dh 64), where two rows share
// the 64 banks, at kc ^ ((r >> 1) & 7).  Both make those 16 accesses hit
// distinct banks; a fill writes whole rows, which a permutation keeps
// conflict-free.
template <int KCH>
__device__ __forceinline__ int kofs(int r, int kc) {
  const int x = KCH == 16 ? (r & 15) : ((r >> 1) & 7);
  return r * KCH * 8 + ((kc ^ x) << 3);
}

// V^T tile: row d holds the 64 keys of dim d (128 bytes, 8 chunks of 8 keys).
// The P.V MFMA of k step s takes, in lane half h, the keys 16s + 4h + {0..3}
// and 16s + 8 + 4h + {0..3}; storing each 16-key group in the order
// [0-3, 8-11, 4-7, 12-15] makes those 8 keys one contiguous chunk (2s + h), read
// with one 128-bit access.  Chunk c of row d lives at chunk c ^ vswz(d).
__device__ __forceinline__ int vswz(int d) { return (d ^ (d >> 3)) & 7; }
// element offset (in bf16) of key k of dim d inside the V^T tile
__device__ __forceinline__ int vofs(int d, int k) {
  const int s = k >> 4, a = (k >> 2) & 3, i = k & 3;
  const int chunk = 2 * s + (a & 1), elem = (a >> 1) * 4 + i;
  return d * KT + ((chunk ^ vswz(d)) << 3) + elem;
}

template <int DH, int NW, int QB, bool OUT_F32>
__global__ void __launch_bounds__(NW * kWave)
    attn_kernel(AttnArgs a, int CQ, int wg_per_group) {
  constexpr int NT = NW * kWave;
  constexpr int QR = 32 * QB;                   // query rows per wave
  constexpr int KCH = DH / 8;                  // 16-byte chunks per key row
  constexpr int K_PER = KT * KCH / NT;          // K chunks per thread per tile
  constexpr int VBLK = (KT / 2) * KCH;          // (2 keys x 8 dims) V blocks per tile
  constexpr int V_PER = (VBLK + NT - 1) / NT;   // ... per thread (the last round may be partial)
  static_assert(K_PER * NT == KT * KCH, "tile/thread mismatch");
  constexpr int NB = DH / 32;                   // 32-wide dim blocks of the output

  __shared__ __attribute__((aligned(16))) bf16 Ks[2][KT * DH];
  __shared__ __attribute__((aligned(16))) bf16 Vt[2][DH * KT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, c = lane & 31;

  const int lid = xcd_remap(blockIdx.x, gridDim.x);
  const int g = lid / wg_per_group, wgi = lid % wg_per_group;
  const int G = a.Hq / a.Hkv;
  const int per_req = G * CQ;                   // chunks per request
  const int total = a.B * per_req;
  const int c0 = wgi * NW;
  const int c_last = min(c0 + NW, total) - 1;
  const int b_lo = c0 / per_req, b_hi = c_last / per_req;

  // this wave's chunk
  const int my = c0 + wave;
  const bool active = my < total;
  const int cc = active ? my : c_last;
  const int b = cc / per_req;
  const int rem = cc - b * per_req;
  const int hq = g * G + rem / CQ;
  const int i0 = (rem % CQ) * QR;

  // Q^T fragments of query block qb: lane supplies Q[row i0 + 32qb + c][dims
  // 16kk + 8*half .. +8]
  bf16x8 qf[QB][DH / 16];
  bool row_ok[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qrow = i0 + 32 * qb + c;
    row_ok[qb] = active && qrow < a.n_s;
    const bf16* qp = (const bf16*)a.q + b * a.q_sb + hq * a.q_sh + (long)(row_ok[qb] ? qrow : 0) * a.q_sr;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok[qb]) v = *reinterpret_cast<const u32x4*>(qp + kk * 16 + half * 8);
      qf[qb][kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int TP = cdiv(a.m, KT), TS = cdiv(a.n_s, KT);
  const int n_tiles = TP + (b_hi - b_lo + 1) * TS;

  // tile t -> (K rows, V rows, row stride, valid keys, owning request or -1)
  auto tile_src = [&](int t, const bf16*& kb, const bf16*& vb, long& rs, int& nv, int& owner) __attribute__((always_inline)) {
    if (t < TP) {
      kb = (const bf16*)a.kp + g * a.p_sh + (long)t * KT * DH;
      vb = (const bf16*)a.vp + g * a.p_sh + (long)t * KT * DH;
      rs = DH;
      nv = min(KT, a.m - t * KT);
      owner = -1;
    } else {
      const int u = t - TP, rb = b_lo + u / TS, tt = u % TS;
      const long off = rb * a.s_sb + g * a.s_sh + (long)tt * KT * a.s_sr;
      kb = (const bf16*)a.ks + off;
      vb = (const bf16*)a.vs + off;
      rs = a.s_sr;
      nv = min(KT, a.n_s - tt * KT);
      owner = rb;
    }
  };

  // Each thread loads K_PER 16-byte K chunks and V_PER pairs of V rows per
  // tile.  Its element offsets inside a tile depend only on the row stride
  // (dh for the prefix, s_sr for a suffix), so they are computed once; a tile
  // adds its scalar base.  In a partial tile rows past the valid keys re-read
  // the tile's first row (always in bounds) and are zeroed when stashed.
  int koff_p[K_PER], koff_s[K_PER], voff_p[V_PER], voff_s[V_PER];
#pragma unroll
  for (int p = 0; p < K_PER; ++p) {
    const int q = tid + p * NT, r = q / KCH, kc = q % KCH;
    koff_p[p] = r * DH + kc * 8;
    koff_s[p] = r * (int)a.s_sr + kc * 8;
  }
#pragma unroll
  for (int p = 0; p < V_PER; ++p) {
    const int q = tid + p * NT, dg = q % KCH, kp = q / KCH;
    const int r0 = q < VBLK ? 2 * kp : 0;
    voff_p[p] = r0 * DH + dg * 8;
    voff_s[p] = r0 * (int)a.s_sr + dg * 8;
  }

  u32x4 kreg[K_PER], vreg[V_PER][2];
  int nv_next = 0;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  auto fetch = [&](int t) __attribute__((always_inline)) {
    const bf16 *kb, *vb;
    long rs;
    int owner;
    tile_src(t, kb, vb, rs, nv_next, owner);
    const bool pre = t < TP;
    if (nv_next == KT) {
#pragma unroll
      for (int p = 0; p < K_PER; ++p)
        kreg[p] = *reinterpret_cast<const u32x4*>(kb + (pre ? koff_p[p] : koff_s[p]));
#pragma unroll
      for (int p = 0; p < V_PER; ++p) {
        const bf16* vp = vb + (pre ? voff_p[p] : voff_s[p]);
        vreg[p][0] = *reinterpret_cast<const u32x4*>(vp);
        vreg[p][1] = *reinterpret_cast<const u32x4*>(vp + rs);
      }
    } else {
#pragma unroll
      for (int p = 0; p < K_PER; ++p) {
        const int q = tid + p * NT, r = q / KCH, kc = q % KCH;
        kreg[p] = *reinterpret_cast<const u32x4*>(kb + (r < nv_next ? r : 0) * rs + kc * 8);
      }
#pragma unroll
      for (int p = 0; p < V_PER; ++p) {
        const int q = tid + p * NT, dg = q % KCH, kp = q / KCH;
        const int r0 = q < VBLK ? 2 * kp : 0;
        vreg[p][0] = *reinterpret_cast<const u32x4*>(vb + (r0 < nv_next ? r0 : 0) * rs + dg * 8);
        vreg[p][1] = *reinterpret_cast<const u32x4*>(vb + (r0 + 1 < nv_next ? r0 + 1 : 0) * rs + dg * 8);
      }
    }
  };
  auto stash = [&](int buf) __attribute__((always_inline)) {
    if (nv_next < KT) {  // partial tile: zero the rows past the valid keys
#pragma unroll
      for (int p = 0; p < K_PER; ++p) {
        const int r = (tid + p * NT) / KCH;
        if (r >= nv_next) kreg[p] = zero4;
      }
#pragma unroll
      for (int p = 0; p < V_PER; ++p) {
        const int kp = (tid + p * NT) / KCH;
        if (2 * kp >= nv_next) vreg[p][0] = zero4;
        if (2 * kp + 1 >= nv_next) vreg[p][1] = zero4;
      }
    }
#pragma unroll
    for (int p = 0; p < K_PER; ++p) {
      const int q = tid + p * NT, r = q / KCH, kc = q % KCH;
      *reinterpret_cast<u32x4*>(&Ks[buf][kofs<KCH>(r, kc)]) = kreg[p];
    }
#pragma unroll
    for (int p = 0; p < V_PER; ++p) {
      const int q = tid + p * NT, dg = q % KCH, kp = q / KCH;
      if (q >= VBLK) continue;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // dim dg*8 + e of keys 2kp (low half) and 2kp+1 (high half), adjacent in V^T
        const uint32_t w = __builtin_amdgcn_perm(vreg[p][1][e >> 1], vreg[p][0][e >> 1],
                                                 (e & 1) ? 0x07060302u : 0x05040100u);
        *reinterpret_cast<uint32_t*>(&Vt[buf][vofs(dg * 8 + e, 2 * kp)]) = w;
      }
    }
  };

  f32x16 o[QB][NB];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) o[qb][nb] = zero16();
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
  }
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  // Pipeline: registers hold tile t+1 while tile t computes; they are written
  // to the other LDS buffer between tile t's S = K.Q^T and its softmax (that
  // buffer was last read in tile t-1, before the previous barrier) and tile
  // t+2 is fetched right after, so its loads have a whole tile to arrive.
  fetch(0);
  stash(0);
  if (n_tiles > 1) fetch(1);
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    int owner, nv;
    {
      const bf16 *kb, *vb;
      long rs;
      tile_src(t, kb, vb, rs, nv, owner);
    }
    const bool mine = active && (owner < 0 || owner == b);
    // ---- S^T = K . Q^T over this tile's 64 keys; each K fragment feeds QB MFMAs
    // (the first k step starts from a zero accumulator operand)
    f32x16 sc[QB][KT / 32];
    if (mine) {
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk)
#pragma unroll
        for (int kb = 0; kb < KT / 32; ++kb) {
          const int r = kb * 32 + c;
          const bf16x8 kf =
              *reinterpret_cast<const bf16x8*>(&Ks[buf][kofs<KCH>(r, kk * 2 + half)]);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            sc[qb][kb] = mfma_32x32x16(kf, qf[qb][kk], kk == 0 ? zero16() : sc[qb][kb]);
        }
    }
    if (t + 1 < n_tiles) {
      stash(buf ^ 1);
      if (t + 2 < n_tiles) fetch(t + 2);
    }
    if (mine) {
      if (nv < KT) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int key = kb * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
              if (key >= nv) sc[qb][kb][e] = -INFINITY;
            }
      }
      // ---- online softmax (log2 domain), one query row per lane per block
      bf16x8 pf[QB][KT / 16];
      const bf16x2 ones = {(bf16)1.f, (bf16)1.f};
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[qb][kb][e]);
        mx = half_max(mx) * sl2;
        // The running max only moves when a row's tile max exceeds it by more
        // than 8 (log2 units): probabilities then stay <= 2^8, exact in fp32
        // and representable in bf16, and the O / l rescale is skipped on most
        // tiles.
        if (__builtin_amdgcn_ballot_w64(mx > m_run[qb] + 8.f)) {
          const float m_new = fmaxf(m_run[qb], mx);
          const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
          l_run[qb] *= alpha;
          m_run[qb] = m_new;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[qb][nb][e] *= alpha;
        }
        // P^T operand of k step s: slot (half, e) is key 16s + 8*(e/4) +
        // 4*half + e%4, i.e. score register 8*(s%2) + e of block s/2.  The row
        // sum accumulates the same bf16-rounded probabilities that the P.V
        // product uses (v_dot2 against (1, 1)); each dot2 takes its packed pair
        // as its own value (taken back out of the 4-dword vector, the compiler
        // feeds every dot2 the first element's register).
#pragma unroll
        for (int s = 0; s < KT / 16; ++s) {
          uint32_t pw[4];
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int e0 = 8 * (s & 1) + 2 * w;
            const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[qb][s >> 1][e0], sl2, -m_run[qb]));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[qb][s >> 1][e0 + 1], sl2, -m_run[qb]));
            const bf16x2 pp = {(bf16)p0, (bf16)p1};
            l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l_run[qb], false);
            pw[w] = __builtin_bit_cast(uint32_t, pp);
          }
          const u32x4 pv = {pw[0], pw[1], pw[2], pw[3]};
          pf[qb][s] = __builtin_bit_cast(bf16x8, pv);
        }
      }

      // ---- O^T += V^T . P^T, 16 keys per MFMA; each V^T fragment feeds QB MFMAs
#pragma unroll
      for (int s = 0; s < KT / 16; ++s) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int r = nb * 32 + c;
          const bf16x8 vf =
              *reinterpret_cast<const bf16x8*>(&Vt[buf][r * KT + (((2 * s + half) ^ vswz(r)) << 3)]);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][nb] = mfma_32x32x16(vf, pf[qb][s], o[qb][nb]);
        }
      }
    }
    __syncthreads();
  }

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (!row_ok[qb]) continue;
    const int qrow = i0 + 32 * qb + c;
    const float l_tot = half_sum(l_run[qb]);
    const float inv = 1.f / l_tot;
    // lane holds O[row][dims nb*32 + 8j + 4*half + i], i = 0..3
    if constexpr (OUT_F32) {
      float* op = (float*)a.out + b * a.o_sb + hq * a.o_sh + (long)qrow * a.o_sr;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f32x4 v = {o[qb][nb][4 * j] * inv, o[qb][nb][4 * j + 1] * inv, o[qb][nb][4 * j + 2] * inv,
                     o[qb][nb][4 * j + 3] * inv};
          *reinterpret_cast<f32x4*>(op + nb * 32 + 8 * j + 4 * half) = v;
        }
    } else {
      bf16* op = (bf16*)a.out + b * a.o_sb + hq * a.o_sh + (long)qrow * a.o_sr;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          u32x2 v = {pack_bf16x2(o[qb][nb][4 * j] * inv, o[qb][nb][4 * j + 1] * inv),
                     pack_bf16x2(o[qb][nb][4 * j + 2] * inv, o[qb][nb][4 * j + 3] * inv)};
          *reinterpret_cast<u32x2*>(op + nb * 32 + 8 * j + 4 * half) = v;
        }
    }
  }
}

template <int DH, int NW, int QB, bool F32>
hipError_t launch_cfg(const AttnArgs& a, hipStream_t s) {
  const int CQ = cdiv(a.n_s, 32 * QB);
  const int G = a.Hq / a.Hkv;
  const int wpg = cdiv(a.B * G * CQ, NW);
  const int grid = a.Hkv * wpg;
  hipLaunchKernelGGL((attn_kernel<DH, NW, QB, F32>), dim3(grid), dim3(NW * kWave), 0, s, a, CQ, wpg);
  return hipGetLastError();
}

// 8 waves x 32 query rows per workgroup
template <int DH, bool F32>
hipError_t launch_dh(const AttnArgs& a, hipStream_t s) {
  return launch_cfg<DH, 8, 1, F32>(a, s);
}

}  // namespace

hipError_t attention(const AttnArgs& a, hipStream_t s) {
  if (a.dh == 128) return a.out_f32 ? launch_dh<128, true>(a, s) : launch_dh<128, false>(a, s);
  return a.out_f32 ? launch_dh<64, true>(a, s) : launch_dh<64, false>(a, s);
}

}  // namespace bc
