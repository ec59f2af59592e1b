// bf16 GEMMs on gfx950 MFMA with the epilogues of the transformer layer:
// residual add (O and down projections), SwiGLU (gate/up projection) and the
// fused Q/K/V projection with optional bias, rotate-half RoPE and head-major
// scatter (which,
// during populate, writes the prefix K/V straight into the cache entry).
//
// C[M, N] = A[M, K] . W[N, K]^T.  Both operands are K-contiguous, so every
// MFMA operand fragment is one 16-byte LDS read per lane and no transpose is
// needed anywhere.
//
// Tiling: a workgroup computes a 256 x 256 tile with 8 waves, each a 64 x 128
// sub-tile of 32x32 MFMA blocks (v_mfma_f32_32x32x16_bf16); K advances in
// steps of 64 through a double-buffered LDS tile pair (see gemm_pp_kernel for
// the schedule).  LDS rows are 128 bytes (64 bf16) with an XOR-swizzled
// 16-byte chunk index (see swz), conflict-free for both the fills and the
// fragment reads.
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
  int w_bytes;  // bytes of W that an epilogue's rows span (its buffer range)
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

// R += A . W^T: the accumulators start from the residual tile (init), so the
// residual is read while the first K steps load and the epilogue only writes.
struct EpiResidual {
  float* R;
  int ldr, N;
  static constexpr bool kInit = true;
  __host__ __device__ int tiles_n(int BN) const { return cdiv(N, BN); }
  __host__ __device__ int w_rows() const { return N; }
  template <int BN, int TN>
  __device__ __forceinline__ int w_row(int tn, int r) const {
    int n = tn * BN + r;
    return n < N ? n : -1;
  }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void init(f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn, int lane) const {
    const int col0 = tn * BN + wn * TN + (lane & 31);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = row0 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const float* rp = R + (long)(row < M ? row : 0) * ldr;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = col0 + j * 32;
          acc[i][j][e] = (row < M && col < N) ? rp[col] : 0.f;
        }
      }
  }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
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
          if (col < N) rp[col] = acc[i][j][e];
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
  static constexpr bool kInit = false;
  __host__ __device__ int tiles_n(int BN) const { return cdiv(F, BN / 2); }
  __host__ __device__ int w_rows() const { return 2 * F; }
  template <int BN, int TN>
  __device__ __forceinline__ int w_row(int tn, int r) const {
    const int wn = r / TN, q = r % TN;
    const int half = q / (TN / 2), within = q % (TN / 2);
    const int col = tn * (BN / 2) + wn * (TN / 2) + within;
    return col < F ? half * F + col : -1;
  }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
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
  static constexpr bool kInit = false;
  bf16* q;
  bf16* k;
  bf16* v;
  long q_sb, q_sh, k_sb, k_sh, v_sb, v_sh;
  int Hq, Hkv, n_seq, pos0;
  const float* cos_t;
  const float* sin_t;
  const bf16* bias;  // [(Hq + 2*Hkv) * DH] added before RoPE, or null
  __host__ __device__ int ncols() const { return (Hq + 2 * Hkv) * DH; }
  __host__ __device__ int tiles_n(int BN) const { return cdiv(ncols(), BN); }
  __host__ __device__ int w_rows() const { return ncols(); }
  template <int BN, int TN>
  __device__ __forceinline__ int w_row(int tn, int r) const {
    int n = tn * BN + r;
    return n < ncols() ? n : -1;
  }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
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
            float x1 = acc[i][hh * BPH + jj][e];
            float x2 = acc[i][hh * BPH + jj + BPH / 2][e];
            if (bias) {
              x1 += bf16_to_f32(bias[head_g * DH + d1]);
              x2 += bf16_to_f32(bias[head_g * DH + d1 + DH / 2]);
            }
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

// ---------------------------------------------------------------- ping-pong kernel
// Same 256 x 256 tile and 64 x 128 wave sub-tiles, but the two waves that
// share a SIMD never do the same kind of work at the same time.  Waves 0-3
// (group 0, columns 0-127 of the tile) and waves 4-7 (group 1, columns
// 128-255) run the same program, group 1 one barrier-phase behind.  Each half
// K step (32 of K) is a memory phase -- read this half step's fragments from
// LDS, write half of the next K step's tile into the free LDS buffer and
// issue the global loads of the same half of the K step after it -- then a
// compute phase of 16 MFMAs, with a workgroup barrier between phases.  While
// one group issues its MFMAs the other group's LDS and global traffic runs,
// so the matrix pipe of every SIMD is fed alternately by its two waves, and
// both memory phases carry the same load.
//
// LDS tiles are double-buffered: K step k+1 is written during step k (after
// every wave has finished reading that buffer's previous tile, step k-1) and
// is first read at step k+1.  Group 0 fetches and writes the A tile, group 1
// the W tile, 8 chunks of 16 bytes per lane per K step, through buffer loads:
// A's descriptor starts at the tile's first row and covers its valid rows, W
// rows that an epilogue maps to nothing get an offset past W's end, so rows
// outside the matrices read as zero with no selects.  Each load has four
// phases (one K step) to land before its chunk is written to LDS.
template <class Epi>
__global__ void __launch_bounds__(512) gemm_pp_kernel(GemmArgs a, Epi epi) {
  constexpr int BM = 256, BN = 256, TM = 64, TN = 128, FM = 2, FN = 4;
  constexpr int PER = 8, HPER = 4;  // 16-byte chunks per lane per K step, per half
  constexpr int RSRC_W3 = 0x00020000;  // raw buffer, 32-bit dwords (gfx9 family)
  constexpr uint32_t kNoRow = 0x80000000u;  // offset past every descriptor's range

  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * BK];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;          // 0: loads A, computes columns 0-127; 1: W, 128-255
  const int wm = wave & 3, wn = grp;  // the two waves on a SIMD are w and w + 4

  const int tiles_m = cdiv(a.M, BM), tiles_n = epi.tiles_n(BN);
  const int lid = xcd_remap(blockIdx.x, gridDim.x);
  // Tile order: each die takes a contiguous range of tiles, swept in groups
  // of GM row tiles, column-major inside a group, so the 32 tiles a die runs
  // at once share A and W panels in its L2.  When a row of tiles is at most
  // 32 wide (the O and down projections: N = h), whole rows run at once
  // (GM = 1): every A panel is then read from HBM once and the small W is
  // re-read from the last-level cache (measured +2% and +4% on the O and down
  // shapes against GM = 8, which suits the wide QKV and gate/up outputs).
  const int GM = tiles_n <= 32 ? 1 : 8;
  const int per_group = GM * tiles_n;
  const int first_m = (lid / per_group) * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int tm = first_m + (lid % per_group) % gsz;
  const int tn = (lid % per_group) / gsz;
  const int m0 = tm * BM;

  // this lane's chunks of its group's operand tile: chunk p covers tile row
  // lane/8 + 8*wm + 32*p, 16-byte column chunk lane%8
  const int kc = lane & 7;
  uint32_t voff[PER];
  __amdgpu_buffer_rsrc_t rsrc;
  if (grp == 0) {
    const int rows = min(BM, a.M - m0);
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(a.A + (long)m0 * a.lda), (short)0,
                                             rows * a.lda * 2, RSRC_W3);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int r = (lane >> 3) + 8 * wm + 32 * p;
      voff[p] = r < rows ? (uint32_t)(r * a.lda + kc * 8) * 2u : kNoRow;
    }
  } else {
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(a.W), (short)0, a.w_bytes, RSRC_W3);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int r = (lane >> 3) + 8 * wm + 32 * p;
      const int gr = epi.template w_row<BN, TN>(tn, r);
      voff[p] = gr >= 0 ? (uint32_t)(gr * a.ldw + kc * 8) * 2u : kNoRow;
    }
  }
  bf16* const dst0 = grp == 0 ? &sA[0][0] : &sB[0][0];
  u32x4 stage[PER];
  auto fetch = [&](int k0, int h) __attribute__((always_inline)) {
#pragma unroll
    for (int p = h * HPER; p < (h + 1) * HPER; ++p)
      stage[p] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff[p], k0 * 2, 0);
  };
  auto stash = [&](int buf, int h) __attribute__((always_inline)) {
    bf16* dst = dst0 + buf * (BM * BK);
#pragma unroll
    for (int p = h * HPER; p < (h + 1) * HPER; ++p) {
      const int r = (lane >> 3) + 8 * wm + 32 * p;
      *reinterpret_cast<u32x4*>(&dst[swz(r, kc)]) = stage[p];
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = zero16();

  bf16x8 fa[2][FM], fb[2][FN];
  auto read_frags = [&](int cur, int h) __attribute__((always_inline)) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int kci = (2 * h + k2) * 2 + (lane >> 5);
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[k2][i] = *reinterpret_cast<const bf16x8*>(&sA[cur][swz(wm * TM + i * 32 + (lane & 31), kci)]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[k2][j] = *reinterpret_cast<const bf16x8*>(&sB[cur][swz(wn * TN + j * 32 + (lane & 31), kci)]);
    }
  };
  auto mma = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma_32x32x16(fa[k2][i], fb[k2][j], acc[i][j]);
  };

  // A phase boundary: the workgroup barrier, fenced so that the compiler
  // cannot move MFMAs (which touch no memory) across it.
  auto phase = []() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
  };

  const int ksteps = a.K / BK;
  // prologue: K step 0 in LDS, K step 1 in the stage registers
  fetch(0, 0);
  fetch(0, 1);
  if constexpr (Epi::kInit) epi.template init<BN, TN, FM, FN>(acc, a.M, tn, m0 + wm * TM, wn, lane);
  stash(0, 0);
  stash(0, 1);
  if (ksteps > 1) {
    fetch(BK, 0);
    fetch(BK, 1);
  }
  phase();
  if (grp == 1) phase();  // group 1 runs one phase behind

  for (int ks = 0; ks < ksteps; ++ks) {
    const int cur = ks & 1;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      read_frags(cur, h);
      if (ks + 1 < ksteps) {
        stash(cur ^ 1, h);
        if (ks + 2 < ksteps) fetch((ks + 2) * BK, h);
      }
      phase();
      mma();
      phase();
    }
  }
  if (grp == 0) phase();  // match group 1's extra barrier

  epi.template apply<BN, TN, FM, FN>(acc, a.M, tn, m0 + wm * TM, wn, lane);
}

// 256 x 256 tiles, 8 waves as 4 (M) x 2 (N): 64 x 128 per wave, so a wave's
// columns span whole 128-wide heads (RoPE pairs stay lane-local).
constexpr int kBM = 256, kBN = 256, kWM = 4, kWN = 2;

template <class Epi>
hipError_t launch(GemmArgs a, const Epi& epi, hipStream_t s) {
  const int tiles = cdiv(a.M, 256) * epi.tiles_n(256);
  if (tiles == 0) return hipSuccess;
  // operand offsets are 32-bit buffer offsets: W and a 256-row A panel must
  // stay below 2 GiB, and K must be whole 64-wide steps
  const long w_bytes = (long)epi.w_rows() * a.ldw * 2, a_panel = 256L * a.lda * 2;
  if (w_bytes >= (1L << 31) || a_panel >= (1L << 31) || a.K % BK) return hipErrorInvalidValue;
  a.w_bytes = (int)w_bytes;
  hipLaunchKernelGGL((gemm_pp_kernel<Epi>), dim3(tiles), dim3(512), 0, s, a, epi);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_residual(const void* A, int lda, const void* W, int ldw, int M, int N, int K,
                         float* R, int ldr, hipStream_t s) {
  GemmArgs a{(const bf16*)A, lda, (const bf16*)W, ldw, M, K, 0};
  EpiResidual e{R, ldr, N};
  return launch(a, e, s);
}

hipError_t gemm_swiglu(const void* A, int lda, const void* W, int ldw, int M, int F, int K,
                       void* act, hipStream_t s) {
  GemmArgs a{(const bf16*)A, lda, (const bf16*)W, ldw, M, K, 0};
  EpiSwiGLU e{(bf16*)act, F};
  return launch(a, e, s);
}

hipError_t gemm_qkv_rope(const void* A, int lda, const void* W, int ldw, int M, int K, int Hq,
                         int Hkv, int dh, int n_seq, int pos0, const float* cos_t,
                         const float* sin_t, const QkvOut& o, hipStream_t s) {
  GemmArgs a{(const bf16*)A, lda, (const bf16*)W, ldw, M, K, 0};
  if (dh == 128) {
    EpiQKV<128> e{(bf16*)o.q, (bf16*)o.k, (bf16*)o.v, o.q_sb, o.q_sh, o.k_sb, o.k_sh,
                  o.v_sb, o.v_sh, Hq, Hkv, n_seq, pos0, cos_t, sin_t, (const bf16*)o.bias};
    return launch(a, e, s);
  }
  EpiQKV<64> e{(bf16*)o.q, (bf16*)o.k, (bf16*)o.v, o.q_sb, o.q_sh, o.k_sb, o.k_sh,
               o.v_sb, o.v_sh, Hq, Hkv, n_seq, pos0, cos_t, sin_t, (const bf16*)o.bias};
  return launch(a, e, s);
}

}  // namespace bc
