// Shared-prefix bidirectional attention on gfx950 (Eq. 2 over [prefix ; own
// suffix], the shallow-layer form of Eq. 4).  With m = 0 the same kernel is
// the deep layers' full attention of every request over its own sequence.
//
// Work decomposition.  For one KV head g, the query rows of every request b
// and every query head of g's group are cut into 32-row chunks (b, head, i0);
// a workgroup of NW waves takes NW consecutive chunks, one per wave.  The key
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
constexpr int QR = 32;  // query rows per wave

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

// V^T rows hold 64 keys = 16 units of 4 keys (8 bytes).  Unit u of row r lives
// at unit u ^ vswz(r): 16 consecutive rows read at the same unit hit 16
// different bank pairs.
__device__ __forceinline__ int vswz(int r) { return (r ^ (r >> 3)) & 15; }

template <int DH, int NW, bool OUT_F32>
__global__ void __launch_bounds__(NW * kWave)
    attn_kernel(AttnArgs a, int CQ, int wg_per_group) {
  constexpr int NT = NW * kWave;
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
  const int qrow = i0 + c;
  const bool row_ok = active && qrow < a.n_s;

  // Q^T fragments: lane supplies Q[row c][dims 16kk + 8*half .. +8]
  bf16x8 qf[DH / 16];
  {
    const bf16* qp = (const bf16*)a.q + b * a.q_sb + hq * a.q_sh + (long)(row_ok ? qrow : 0) * a.q_sr;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row_ok) v = *reinterpret_cast<const u32x4*>(qp + kk * 16 + half * 8);
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int TP = cdiv(a.m, KT), TS = cdiv(a.n_s, KT);
  const int n_tiles = TP + (b_hi - b_lo + 1) * TS;

  // tile t -> (K rows, V rows, row stride, valid keys, owning request or -1)
  auto tile_src = [&](int t, const bf16*& kb, const bf16*& vb, long& rs, int& nv, int& owner) {
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

  u32x4 kreg[K_PER], vreg[V_PER][2];
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  auto fetch = [&](int t) {
    const bf16 *kb, *vb;
    long rs;
    int nv, owner;
    tile_src(t, kb, vb, rs, nv, owner);
#pragma unroll
    for (int p = 0; p < K_PER; ++p) {
      const int q = tid + p * NT, r = q / KCH, kc = q % KCH;
      kreg[p] = r < nv ? *reinterpret_cast<const u32x4*>(kb + r * rs + kc * 8) : zero4;
    }
#pragma unroll
    for (int p = 0; p < V_PER; ++p) {
      const int q = tid + p * NT, dg = q % KCH, kp = q / KCH;
      const int r0 = q < VBLK ? 2 * kp : KT;
      vreg[p][0] = r0 < nv ? *reinterpret_cast<const u32x4*>(vb + r0 * rs + dg * 8) : zero4;
      vreg[p][1] = r0 + 1 < nv ? *reinterpret_cast<const u32x4*>(vb + (r0 + 1) * rs + dg * 8) : zero4;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int p = 0; p < K_PER; ++p) {
      const int q = tid + p * NT, r = q / KCH, kc = q % KCH;
      *reinterpret_cast<u32x4*>(&Ks[buf][r * DH + ((kc ^ (r & 7)) << 3)]) = kreg[p];
    }
#pragma unroll
    for (int p = 0; p < V_PER; ++p) {
      const int q = tid + p * NT, dg = q % KCH, kp = q / KCH;
      if (q >= VBLK) continue;
      const int unit = kp >> 1, sub = kp & 1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = dg * 8 + e;
        // keys 2kp (low half) and 2kp+1 (high half) of dim d
        const uint32_t lo = (vreg[p][0][e >> 1] >> ((e & 1) * 16)) & 0xffffu;
        const uint32_t hi = (vreg[p][1][e >> 1] >> ((e & 1) * 16)) & 0xffffu;
        *reinterpret_cast<uint32_t*>(&Vt[buf][d * KT + ((unit ^ vswz(d)) << 2) + sub * 2]) =
            lo | (hi << 16);
      }
    }
  };

  f32x16 o[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) o[nb] = zero16();
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;  // scale * log2(e)

  fetch(0);
  stash(0);
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < n_tiles) fetch(t + 1);

    int owner, nv;
    {
      const bf16 *kb, *vb;
      long rs;
      tile_src(t, kb, vb, rs, nv, owner);
    }
    if (active && (owner < 0 || owner == b)) {
      // ---- S^T = K . Q^T over this tile's 64 keys
      f32x16 sc[KT / 32];
#pragma unroll
      for (int kb = 0; kb < KT / 32; ++kb) sc[kb] = zero16();
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk)
#pragma unroll
        for (int kb = 0; kb < KT / 32; ++kb) {
          const int r = kb * 32 + c;
          const bf16x8 kf =
              *reinterpret_cast<const bf16x8*>(&Ks[buf][r * DH + (((kk * 2 + half) ^ (r & 7)) << 3)]);
          sc[kb] = mfma_32x32x16(kf, qf[kk], sc[kb]);
        }
      if (nv < KT) {
#pragma unroll
        for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = kb * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
            if (key >= nv) sc[kb][e] = -INFINITY;
          }
      }
      // ---- online softmax (log2 domain)
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[kb][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float m_new = fmaxf(m_run, mx * sl2);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float lsum = 0.f;
#pragma unroll
      for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sc[kb][e], sl2, -m_new));
          sc[kb][e] = p;
          lsum += p;
        }
      l_run = l_run * alpha + lsum;
      m_run = m_new;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[nb][e] *= alpha;

      // ---- O^T += V^T . P^T, 16 keys per MFMA.  k slot (half, e) of step s
      // is key 16s + 8*(e/4) + 4*half + e%4, which is exactly score register
      // 8*(s%2) + e of block s/2 held by this lane.
#pragma unroll
      for (int s = 0; s < KT / 16; ++s) {
        const int kb = s >> 1, base = 8 * (s & 1);
        u32x4 pw;
#pragma unroll
        for (int w = 0; w < 4; ++w) pw[w] = pack_bf16x2(sc[kb][base + 2 * w], sc[kb][base + 2 * w + 1]);
        const bf16x8 pf = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int r = nb * 32 + c;
          const u32x2 lo = *reinterpret_cast<const u32x2*>(&Vt[buf][r * KT + (((4 * s + half) ^ vswz(r)) << 2)]);
          const u32x2 hi =
              *reinterpret_cast<const u32x2*>(&Vt[buf][r * KT + (((4 * s + 2 + half) ^ vswz(r)) << 2)]);
          const u32x4 vw = {lo[0], lo[1], hi[0], hi[1]};
          o[nb] = mfma_32x32x16(__builtin_bit_cast(bf16x8, vw), pf, o[nb]);
        }
      }
    }
    if (t + 1 < n_tiles) stash(buf ^ 1);
    __syncthreads();
  }

  if (!row_ok) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32, kWave);
  const float inv = 1.f / l_tot;
  // lane holds O[row c][dims nb*32 + 8j + 4*half + i], i = 0..3
  if constexpr (OUT_F32) {
    float* op = (float*)a.out + b * a.o_sb + hq * a.o_sh + (long)qrow * a.o_sr;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f32x4 v = {o[nb][4 * j] * inv, o[nb][4 * j + 1] * inv, o[nb][4 * j + 2] * inv,
                   o[nb][4 * j + 3] * inv};
        *reinterpret_cast<f32x4*>(op + nb * 32 + 8 * j + 4 * half) = v;
      }
  } else {
    bf16* op = (bf16*)a.out + b * a.o_sb + hq * a.o_sh + (long)qrow * a.o_sr;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u32x2 v = {pack_bf16x2(o[nb][4 * j] * inv, o[nb][4 * j + 1] * inv),
                   pack_bf16x2(o[nb][4 * j + 2] * inv, o[nb][4 * j + 3] * inv)};
        *reinterpret_cast<u32x2*>(op + nb * 32 + 8 * j + 4 * half) = v;
      }
  }
}

constexpr int kNW = 8;

template <int DH, bool F32>
hipError_t launch_dh(const AttnArgs& a, hipStream_t s) {
  const int CQ = cdiv(a.n_s, QR);
  const int G = a.Hq / a.Hkv;
  const int wpg = cdiv(a.B * G * CQ, kNW);
  const int grid = a.Hkv * wpg;
  hipLaunchKernelGGL((attn_kernel<DH, kNW, F32>), dim3(grid), dim3(kNW * kWave), 0, s, a, CQ, wpg);
  return hipGetLastError();
}

}  // namespace

hipError_t attention(const AttnArgs& a, hipStream_t s) {
  if (a.dh == 128) return a.out_f32 ? launch_dh<128, true>(a, s) : launch_dh<128, false>(a, s);
  return a.out_f32 ? launch_dh<64, true>(a, s) : launch_dh<64, false>(a, s);
}

}  // namespace bc
