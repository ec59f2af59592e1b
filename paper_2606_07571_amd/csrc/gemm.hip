// bf16 GEMMs on gfx950 MFMA with the epilogues of the transformer layer:
// residual add (O and down projections), SwiGLU (gate/up projection) and the
// fused Q/K/V projection with rotate-half RoPE and head-major scatter (which,
// during populate, writes the prefix K/V straight into the cache entry).
//
// C[M, N] = A[M, K] . W[N, K]^T.  Both operands are K-contiguous, so every
// MFMA operand fragment is one 16-byte LDS read per lane and no transpose is
// needed anywhere.
//
// Tiling: a workgroup computes a BM x BN tile with WM x WN waves; each wave
// owns a (BM/WM) x (BN/WN) sub-tile made of 32x32 MFMA blocks
// (v_mfma_f32_32x32x16_bf16).  K advances in steps of 64 through a
// double-buffered LDS ring fed through registers: step k+1's tiles are written
// to the other LDS buffer halfway through step k's MFMAs and step k+2's global
// loads are issued right after, with one barrier per step.  LDS rows are 128 bytes
// (64 bf16) with an XOR-swizzled 16-byte chunk index (see swz), conflict-free
// for both the fills and the fragment reads.
#include "device_common.hpp"
#include "kernels.hpp"

namespace bc {
namespace {

constexpr int BK = 64;

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

struct GemmArgs {
  const bf16* A;
  int lda;
  const bf16* W;
  int ldw;
  int M, K;
};

// LDS serves 128-bit accesses 16 lanes (256 bytes, 64 banks) at a time; with
// 128-byte rows two consecutive rows fill the 64 banks, so the chunk index is
// XOR-ed with (row >> 1) & 7: the 16 rows read together by a fragment load, and
// the 2 rows x 8 chunks written together by a fill, all land on distinct banks.
__device__ __forceinline__ int swz(int row, int kc) { return row * BK + ((kc ^ ((row >> 1) & 7)) << 3); }

// ---------------------------------------------------------------- epilogues
// Each epilogue says how many BN-wide tiles cover its output (tiles_n), which
// row of W feeds tile-local B row r (w_row, -1 = zero row) and how the wave's
// accumulators are written (apply).  Accumulator (i, j, e) of lane l holds
// C[row0 + i*32 + 8*(e/4) + 4*(l/32) + e%4][col0 + j*32 + l%32].

struct EpiResidual {
  float* R;
  int ldr, N;
  __host__ __device__ int tiles_n(int BN) const { return cdiv(N, BN); }
  template <int BN, int TN>
  __device__ int w_row(int tn, int r) const {
    int n = tn * BN + r;
    return n < N ? n : -1;
  }
  template <int BN, int TN, int FM, int FN>
  __device__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
                        int lane) const {
    const int col0 = tn * BN + wn * TN + (lane & 31);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = row0 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row >= M) continue;
        float* rp = R + (long)row * ldr;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = col0 + j * 32;
          if (col < N) rp[col] += acc[i][j][e];
        }
      }
  }
};

// Gate and up rows of the same output columns are interleaved inside each
// wave's sub-tile: the first TN/2 B rows of a wave are gate rows, the last TN/2
// are the up rows of the same columns, so silu(g) * u is lane-local.
struct EpiSwiGLU {
  bf16* act;
  int F;
  __host__ __device__ int tiles_n(int BN) const { return cdiv(F, BN / 2); }
  template <int BN, int TN>
  __device__ int w_row(int tn, int r) const {
    const int wn = r / TN, q = r % TN;
    const int half = q / (TN / 2), within = q % (TN / 2);
    const int col = tn * (BN / 2) + wn * (TN / 2) + within;
    return col < F ? half * F + col : -1;
  }
  template <int BN, int TN, int FM, int FN>
  __device__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
                        int lane) const {
    const int col0 = tn * (BN / 2) + wn * (TN / 2) + (lane & 31);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = row0 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row >= M) continue;
        bf16* op = act + (long)row * F;
#pragma unroll
        for (int j = 0; j < FN / 2; ++j) {
          const int col = col0 + j * 32;
          if (col >= F) continue;
          const float g = acc[i][j][e], u = acc[i][j + FN / 2][e];
          op[col] = to_bf16(g / (1.f + __expf(-g)) * u);
        }
      }
  }
};

template <int DH>
struct EpiQKV {
  bf16* q;
  bf16* k;
  bf16* v;
  long q_sb, q_sh, k_sb, k_sh, v_sb, v_sh;
  int Hq, Hkv, n_seq, pos0;
  const float* cos_t;
  const float* sin_t;
  __host__ __device__ int ncols() const { return (Hq + 2 * Hkv) * DH; }
  __host__ __device__ int tiles_n(int BN) const { return cdiv(ncols(), BN); }
  template <int BN, int TN>
  __device__ int w_row(int tn, int r) const {
    int n = tn * BN + r;
    return n < ncols() ? n : -1;
  }
  template <int BN, int TN, int FM, int FN>
  __device__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
                        int lane) const {
    static_assert(TN % DH == 0, "a wave sub-tile must hold whole heads");
    constexpr int BPH = DH / 32;  // 32-column blocks per head
#pragma unroll
    for (int hh = 0; hh < TN / DH; ++hh) {
      const int head_g = (tn * BN + wn * TN) / DH + hh;
      if (head_g >= Hq + 2 * Hkv) continue;
      bf16* base;
      long sb, sh;
      int head;
      bool rot = true;
      if (head_g < Hq) {
        base = q; sb = q_sb; sh = q_sh; head = head_g;
      } else if (head_g < Hq + Hkv) {
        base = k; sb = k_sb; sh = k_sh; head = head_g - Hq;
      } else {
        base = v; sb = v_sb; sh = v_sh; head = head_g - Hq - Hkv; rot = false;
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = row0 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (row >= M) continue;
          const int b = row / n_seq, t = row - b * n_seq;
          bf16* dst = base + b * sb + head * sh + (long)t * DH;
          const float* ct = cos_t + (long)(pos0 + t) * (DH / 2);
          const float* st = sin_t + (long)(pos0 + t) * (DH / 2);
#pragma unroll
          for (int jj = 0; jj < BPH / 2; ++jj) {
            const int d1 = jj * 32 + (lane & 31);
            const float x1 = acc[i][hh * BPH + jj][e];
            const float x2 = acc[i][hh * BPH + jj + BPH / 2][e];
            float y1 = x1, y2 = x2;
            if (rot) {
              const float c = ct[d1], s = st[d1];
              y1 = x1 * c - x2 * s;
              y2 = x2 * c + x1 * s;
            }
            dst[d1] = to_bf16(y1);
            dst[d1 + DH / 2] = to_bf16(y2);
          }
        }
    }
  }
};

// ---------------------------------------------------------------- kernel

template <int BM, int BN, int WM, int WN, class Epi>
__global__ void __launch_bounds__(WM * WN * kWave) gemm_kernel(GemmArgs a, Epi epi) {
  constexpr int NT = WM * WN * kWave;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int A_PER = BM * BK / 8 / NT;  // 16-byte chunks per thread per step
  constexpr int B_PER = BN * BK / 8 / NT;
  static_assert(A_PER * NT * 8 == BM * BK && B_PER * NT * 8 == BN * BK, "tile/thread mismatch");

  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * BK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // tile order: XCD-contiguous, then groups of 8 row-tiles swept column-major
  const int tiles_m = cdiv(a.M, BM), tiles_n = epi.tiles_n(BN);
  const int lid = xcd_remap(blockIdx.x, gridDim.x);
  constexpr int GM = 8;
  const int per_group = GM * tiles_n;
  const int first_m = (lid / per_group) * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int tm = first_m + (lid % per_group) % gsz;
  const int tn = (lid % per_group) / gsz;
  const int m0 = tm * BM;

  // per-thread chunk sources: chunk p covers tile row tid/8 + p*NT/8, column chunk tid%8
  const int kc = tid & 7;
  const bf16* a_src[A_PER];
  bool a_ok[A_PER];
#pragma unroll
  for (int p = 0; p < A_PER; ++p) {
    const int r = (tid >> 3) + p * (NT / 8);
    const int gr = m0 + r;
    a_ok[p] = gr < a.M;
    a_src[p] = a.A + (long)(a_ok[p] ? gr : 0) * a.lda + kc * 8;
  }
  const bf16* b_src[B_PER];
  bool b_ok[B_PER];
#pragma unroll
  for (int p = 0; p < B_PER; ++p) {
    const int r = (tid >> 3) + p * (NT / 8);
    const int wr = epi.template w_row<BN, TN>(tn, r);
    b_ok[p] = wr >= 0;
    b_src[p] = a.W + (long)(b_ok[p] ? wr : 0) * a.ldw + kc * 8;
  }

  u32x4 ra[A_PER], rb[B_PER];
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  // Loads are unconditional (an invalid row reads the clamped row 0, always in
  // bounds) so that no load sits behind a divergent branch; rows outside the
  // matrix are zeroed only when the registers are written to LDS, after the
  // current step's MFMAs, so the load latency stays hidden behind them.
  auto fetch = [&](int k0) {
#pragma unroll
    for (int p = 0; p < A_PER; ++p) ra[p] = *reinterpret_cast<const u32x4*>(a_src[p] + k0);
#pragma unroll
    for (int p = 0; p < B_PER; ++p) rb[p] = *reinterpret_cast<const u32x4*>(b_src[p] + k0);
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int p = 0; p < A_PER; ++p) {
      const int r = (tid >> 3) + p * (NT / 8);
      *reinterpret_cast<u32x4*>(&sA[buf][swz(r, kc)]) = a_ok[p] ? ra[p] : zero4;
    }
#pragma unroll
    for (int p = 0; p < B_PER; ++p) {
      const int r = (tid >> 3) + p * (NT / 8);
      *reinterpret_cast<u32x4*>(&sB[buf][swz(r, kc)]) = b_ok[p] ? rb[p] : zero4;
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = zero16();

  const int ksteps = a.K / BK;
  auto compute = [&](int cur, int kk0, int kk1) {
#pragma unroll
    for (int kk = kk0; kk < kk1; ++kk) {
      const int kci = kk * 2 + (lane >> 5);
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int r = wm * TM + i * 32 + (lane & 31);
        af[i] = *reinterpret_cast<const bf16x8*>(&sA[cur][swz(r, kci)]);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int r = wn * TN + j * 32 + (lane & 31);
        bfr[j] = *reinterpret_cast<const bf16x8*>(&sB[cur][swz(r, kci)]);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma_32x32x16(af[i], bfr[j], acc[i][j]);
    }
  };

  // Pipeline: the registers hold step ks+1 while step ks computes; they are
  // written to the other LDS buffer halfway through step ks (that buffer was
  // last read in step ks-1, before the previous barrier), and step ks+2 is
  // fetched right after, so its loads have a whole step to arrive and the LDS
  // writes overlap the second half of the step's MFMAs.
  fetch(0);
  stash(0);
  if (ksteps > 1) fetch(BK);
  __syncthreads();

  for (int ks = 0; ks < ksteps; ++ks) {
    const int cur = ks & 1;
    compute(cur, 0, BK / 32);
    if (ks + 1 < ksteps) {
      stash(cur ^ 1);
      if (ks + 2 < ksteps) fetch((ks + 2) * BK);
    }
    compute(cur, BK / 32, BK / 16);
    __syncthreads();
  }

  epi.template apply<BN, TN, FM, FN>(acc, a.M, tn, m0 + wm * TM, wn, lane);
}

// 256 x 256 tiles, 8 waves as 4 (M) x 2 (N): 64 x 128 per wave, so a wave's
// columns span whole 128-wide heads (RoPE pairs stay lane-local).
constexpr int kBM = 256, kBN = 256, kWM = 4, kWN = 2;

template <class Epi>
hipError_t launch(const GemmArgs& a, const Epi& epi, hipStream_t s) {
  const int tiles = cdiv(a.M, kBM) * epi.tiles_n(kBN);
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<kBM, kBN, kWM, kWN, Epi>), dim3(tiles), dim3(kWM * kWN * kWave),
                     0, s, a, epi);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_residual(const void* A, int lda, const void* W, int ldw, int M, int N, int K,
                         float* R, int ldr, hipStream_t s) {
  GemmArgs a{(const bf16*)A, lda, (const bf16*)W, ldw, M, K};
  EpiResidual e{R, ldr, N};
  return launch(a, e, s);
}

hipError_t gemm_swiglu(const void* A, int lda, const void* W, int ldw, int M, int F, int K,
                       void* act, hipStream_t s) {
  GemmArgs a{(const bf16*)A, lda, (const bf16*)W, ldw, M, K};
  EpiSwiGLU e{(bf16*)act, F};
  return launch(a, e, s);
}

hipError_t gemm_qkv_rope(const void* A, int lda, const void* W, int ldw, int M, int K, int Hq,
                         int Hkv, int dh, int n_seq, int pos0, const float* cos_t,
                         const float* sin_t, const QkvOut& o, hipStream_t s) {
  GemmArgs a{(const bf16*)A, lda, (const bf16*)W, ldw, M, K};
  if (dh == 128) {
    EpiQKV<128> e{(bf16*)o.q, (bf16*)o.k, (bf16*)o.v, o.q_sb, o.q_sh, o.k_sb, o.k_sh,
                  o.v_sb, o.v_sh, Hq, Hkv, n_seq, pos0, cos_t, sin_t};
    return launch(a, e, s);
  }
  EpiQKV<64> e{(bf16*)o.q, (bf16*)o.k, (bf16*)o.v, o.q_sb, o.q_sh, o.k_sb, o.k_sh,
               o.v_sb, o.v_sh, Hq, Hkv, n_seq, pos0, cos_t, sin_t};
  return launch(a, e, s);
}

}  // namespace bc
