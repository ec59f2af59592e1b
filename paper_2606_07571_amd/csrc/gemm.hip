// bf16 GEMMs on gfx950 MFMA with the epilogues of the transformer layer:
// residual add (O and down projections), SwiGLU (gate/up projection) and the
// fused Q/K/V projection with optional bias, rotate-half RoPE and head-major
// scatter (which, during populate, writes the prefix K/V straight into the
// cache entry).
//
// C[M, N] = A[M, K] . W[N, K]^T.  Both operands are K-contiguous, so every
// MFMA operand fragment is one 16-byte LDS read per lane and no transpose is
// needed anywhere.
//
// Tiling: a workgroup of 4 waves (one per SIMD) computes a 256 x 256 tile,
// each wave a 128 x 128 sub-tile of 4 x 4 32x32 blocks
// (v_mfma_f32_32x32x16_bf16, accumulators in the 256 accumulation registers).
// K advances in steps of 64 through LDS rings of three A tiles and two W
// tiles (160 KiB); operand tiles are loaded straight into LDS (buffer loads
// with the LDS bit), so no register staging is needed.  LDS rows are 128 bytes (64 bf16) with an XOR-swizzled
// 16-byte chunk index (see swz), conflict-free for the fragment reads.  After
// the K loop the tile buffers become the epilogue's staging area: every
// epilogue writes its outputs as whole 16-byte row chunks.
#include <type_traits>

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
// XOR-ed with (row >> 1) & 7: the 16 rows read together by a fragment load all
// land on distinct banks.
__device__ __forceinline__ int swz(int row, int kc) { return row * BK + ((kc ^ ((row >> 1) & 7)) << 3); }

// ---------------------------------------------------------------- epilogues
// Each epilogue says how many BN-wide tiles cover its output (tiles_n), which
// row of W feeds tile-local B row r (w_row, -1 = zero row) and how a wave's
// accumulators leave (apply).  Accumulator (i, j, e) of lane l holds
// C[row0 + i*32 + 8*(e/4) + 4*(l/32) + e%4][col0 + j*32 + l%32]: a lane holds
// columns, so every epilogue first writes its values to its slot of LDS and
// reads them back as row chunks.  `half` is one of the two 64 KiB halves of
// the tile buffers (shared by two waves), `slot` the wave's index in it.

// R += A . W^T, fp32.  32 rows at a time: the accumulators of a 32-row block go
// to LDS (row pitch 4 TN + 32 bytes, so the two half-waves of a write land on
// disjoint banks), come back as 4-column row chunks, are added to the residual
// chunks (loaded one block ahead) and stored.  Whole chunks with a row stride
// that is a multiple of 4 move as 16-byte vectors, others element by element.
struct EpiResidual {
  float* R;
  int ldr, N;
  __host__ __device__ int tiles_n(int BN) const { return cdiv(N, BN); }
  __host__ __device__ int w_rows() const { return N; }
  template <int BN, int TN>
  __device__ __forceinline__ int w_row(int tn, int r) const {
    int n = tn * BN + r;
    return n < N ? n : -1;
  }
  static constexpr int kSlotBytes(int TN, int) { return 32 * (TN * 4 + 32); }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
                                        int lane, char* half, int slot) const {
    const int colw = tn * BN + wn * TN;
    constexpr int P = TN * 4 + 32;
    char* lds = half + slot * (32 * P);
    constexpr int CPR = TN / 4;    // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;  // rows per instruction
    constexpr int NR = 32 / RPI;   // instructions per 32-row block
    const int cr = lane / CPR, col = colw + (lane % CPR) * 4;
    const bool whole = col + 4 <= N && (ldr & 3) == 0;
    f32x4 rv[2][NR];
    auto load_r = [&](int i, int set) __attribute__((always_inline)) {
#pragma unroll
      for (int n = 0; n < NR; ++n) {
        const int row = row0 + i * 32 + n * RPI + cr;
        const float* rp = R + (long)row * ldr + col;
        f32x4 x = {0.f, 0.f, 0.f, 0.f};
        if (row < M) {
          if (whole) {
            x = *reinterpret_cast<const f32x4*>(rp);
          } else {
#pragma unroll
            for (int u = 0; u < 4; ++u)
              if (col + u < N) x[u] = rp[u];
          }
        }
        rv[set][n] = x;
      }
    };
    load_r(0, 0);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if (i + 1 < FM) load_r(i + 1, (i + 1) & 1);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          *reinterpret_cast<float*>(lds + r * P + (j * 32 + (lane & 31)) * 4) = acc[i][j][e];
      }
#pragma unroll
      for (int n = 0; n < NR; ++n) {
        const int r = n * RPI + cr, row = row0 + i * 32 + r;
        const f32x4 v = *reinterpret_cast<const f32x4*>(lds + r * P + (lane % CPR) * 16) + rv[i & 1][n];
        if (row >= M) continue;
        float* rp = R + (long)row * ldr + col;
        if (whole) {
          *reinterpret_cast<f32x4*>(rp) = v;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (col + u < N) rp[u] = v[u];
        }
      }
    }
  }
};

// act = silu(g) * u, bf16.  Gate and up rows of the same output columns are
// interleaved inside each wave's sub-tile: the first TN/2 B rows of a wave are
// gate rows, the last TN/2 the up rows of the same columns, so the product is
// lane-local.  silu(g) * u = g u / (1 + e^-g) with a hardware reciprocal.  The
// wave's (FM*32) x (TN/2) block goes through LDS (row pitch TN + 16 bytes) and
// leaves as 16-byte stores of 8-column row chunks; a chunk not whole inside F
// (or F not a multiple of 8) is stored element by element.
struct EpiSwiGLU {
  bf16* act;
  int F;
  __host__ __device__ int tiles_n(int BN) const { return cdiv(F, BN / 2); }
  __host__ __device__ int w_rows() const { return 2 * F; }
  template <int BN, int TN>
  __device__ __forceinline__ int w_row(int tn, int r) const {
    const int wn = r / TN, q = r % TN;
    const int half = q / (TN / 2), within = q % (TN / 2);
    const int col = tn * (BN / 2) + wn * (TN / 2) + within;
    return col < F ? half * F + col : -1;
  }
  static constexpr int kSlotBytes(int TN, int TM) { return TM * (TN + 16); }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
                                        int lane, char* half, int slot) const {
    const int colw = tn * (BN / 2) + wn * (TN / 2);
    constexpr int P = TN + 16;
    char* lds = half + slot * (FM * 32 * P);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
#pragma unroll
        for (int j = 0; j < FN / 2; ++j) {
          const float g = acc[i][j][e], u = acc[i][j + FN / 2][e];
          *reinterpret_cast<bf16*>(lds + r * P + (j * 32 + (lane & 31)) * 2) =
              to_bf16(g * u * __builtin_amdgcn_rcpf(1.f + __expf(-g)));
        }
      }
    constexpr int CPR = TN / 16;   // 16-byte chunks per row
    constexpr int RPP = 64 / CPR;  // rows per pass
    const int col = colw + (lane % CPR) * 8;
    const bool whole = col + 8 <= F && (F & 7) == 0;
#pragma unroll
    for (int p = 0; p < FM * 32 / RPP; ++p) {
      const int r = p * RPP + lane / CPR;
      const bf16x8 v = *reinterpret_cast<const bf16x8*>(lds + r * P + (lane % CPR) * 16);
      if (row0 + r >= M) continue;
      bf16* op = act + (long)(row0 + r) * F + col;
      if (whole) {
        *reinterpret_cast<bf16x8*>(op) = v;
      } else {
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (col + u < F) op[u] = v[u];
      }
    }
  }
};

// Q/K/V heads, bf16, head-major.  Output column block j of W (head j, DH rows)
// goes to Q head j (j < Hq), K head j - Hq (j < Hq + Hkv) or V head
// j - Hq - Hkv; the bias (one per column, or null) is added first, then Q and K
// are rotated (rotate-half RoPE: dims i and i + DH/2 form a pair) with the
// fp32 tables cos_t/sin_t [pos][DH/2].  A wave's sub-tile holds whole heads.
// 32 rows at a time go through LDS in fp32 (row pitch 4 TN + 32 bytes); reading
// back, a lane takes 8 rotation pairs (i, i + DH/2) of one row: 16-byte LDS
// reads, 16-byte loads of the cos/sin rows, and two 16-byte bf16 stores
// (element by element if a part's strides are not multiples of 8).
template <int DH>
struct EpiQKV {
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
  static constexpr int kSlotBytes(int TN, int) { return 32 * (TN * 4 + 32); }
  template <int BN, int TN, int FM, int FN>
  __device__ __forceinline__ void apply(const f32x16 (&acc)[FM][FN], int M, int tn, int row0, int wn,
                                        int lane, char* half, int slot) const {
    static_assert(TN % DH == 0 && DH % 16 == 0, "a wave sub-tile must hold whole heads");
    const int col0 = tn * BN + wn * TN;
    const int head0 = col0 / DH;
    const bool vec = ((q_sb | q_sh | k_sb | k_sh | v_sb | v_sh) & 7) == 0;
    constexpr int P = TN * 4 + 32;
    char* lds = half + slot * (32 * P);
    float bj[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int c = col0 + j * 32 + (lane & 31);
      bj[j] = bias && c < ncols() ? bf16_to_f32(bias[c]) : 0.f;
    }
    constexpr int GPH = DH / 16;          // 8-pair groups per head
    constexpr int LPR = (TN / DH) * GPH;  // lanes per row
    constexpr int RPI = 64 / LPR;         // rows per instruction
    const int g = lane % LPR, hh = g / GPH, d0 = (g % GPH) * 8;
    const int c1 = hh * DH + d0, c2 = c1 + DH / 2;
    const int head_g = head0 + hh;
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
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          float x = acc[i][j][e];
          if (bias) x += bj[j];
          *reinterpret_cast<float*>(lds + r * P + (j * 32 + (lane & 31)) * 4) = x;
        }
      }
#pragma unroll
      for (int n = 0; n < 32 / RPI; ++n) {
        const int r = n * RPI + lane / LPR, row = row0 + i * 32 + r;
        const f32x4 a0 = *reinterpret_cast<const f32x4*>(lds + r * P + c1 * 4);
        const f32x4 a1 = *reinterpret_cast<const f32x4*>(lds + r * P + c1 * 4 + 16);
        const f32x4 b0 = *reinterpret_cast<const f32x4*>(lds + r * P + c2 * 4);
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(lds + r * P + c2 * 4 + 16);
        if (row >= M || head_g >= Hq + 2 * Hkv) continue;
        const int b = row / n_seq, t = row - b * n_seq;
        const float x1[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        const float x2[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
        bf16x8 o1, o2;
        if (rot) {
          const float* ct = cos_t + (long)(pos0 + t) * (DH / 2) + d0;
          const float* st = sin_t + (long)(pos0 + t) * (DH / 2) + d0;
          const f32x4 c0 = *reinterpret_cast<const f32x4*>(ct), c4 = *reinterpret_cast<const f32x4*>(ct + 4);
          const f32x4 s0 = *reinterpret_cast<const f32x4*>(st), s4 = *reinterpret_cast<const f32x4*>(st + 4);
          const float cc[8] = {c0.x, c0.y, c0.z, c0.w, c4.x, c4.y, c4.z, c4.w};
          const float ss[8] = {s0.x, s0.y, s0.z, s0.w, s4.x, s4.y, s4.z, s4.w};
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            o1[u] = to_bf16(x1[u] * cc[u] - x2[u] * ss[u]);
            o2[u] = to_bf16(x2[u] * cc[u] + x1[u] * ss[u]);
          }
        } else {
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            o1[u] = to_bf16(x1[u]);
            o2[u] = to_bf16(x2[u]);
          }
        }
        bf16* dst = base + b * sb + head * sh + (long)t * DH + d0;
        if (vec) {
          *reinterpret_cast<bf16x8*>(dst) = o1;
          *reinterpret_cast<bf16x8*>(dst + DH / 2) = o2;
        } else {
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            dst[u] = o1[u];
            dst[u + DH / 2] = o2[u];
          }
        }
      }
    }
  }
};

// ---------------------------------------------------------------- loads into LDS
typedef int i32x4 __attribute__((ext_vector_type(4)));

// 16 bytes per lane from a buffer straight into LDS: lane l's chunk lands at
// LDS byte address M0 + inst_offset + 16 l, and is read from the buffer at
// voffset + soffset + inst_offset (out-of-range offsets read as zero).  Loads
// go in groups of four sharing one M0 value: sub 0 sets M0 (one wait state
// before the load reads it), subs 1-3 add 1, 2, 3 KiB through the instruction
// offset, which the caller has subtracted from their voffset.  Written as
// inline assembly so that the compiler does not count these loads: it would
// otherwise wait for every one of them before any LDS read.  The kernel waits
// for them itself (vmcnt) before the barrier that publishes a tile.  M0 is
// written only here; nothing else in the kernels reads it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void load_lds16(i32x4 rsrc, uint32_t voff, uint32_t soff, uint32_t lds, int sub) {
  switch (sub) {
    case 0:
      asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                   :: "v"(voff), "s"(rsrc), "s"(soff), "s"(lds) : "memory", "m0");
      break;
    case 1:
      asm volatile("buffer_load_dwordx4 %0, %1, %2 offen offset:1024 lds"
                   :: "v"(voff), "s"(rsrc), "s"(soff) : "memory");
      break;
    case 2:
      asm volatile("buffer_load_dwordx4 %0, %1, %2 offen offset:2048 lds"
                   :: "v"(voff), "s"(rsrc), "s"(soff) : "memory");
      break;
    default:
      asm volatile("buffer_load_dwordx4 %0, %1, %2 offen offset:3072 lds"
                   :: "v"(voff), "s"(rsrc), "s"(soff) : "memory");
      break;
  }
}
#pragma clang diagnostic pop

// Wait for this wave's LDS reads and for all (or all but the 8 newest) of its
// loads into LDS, then the workgroup barrier, in one statement so that no LDS
// access moves across it.
__device__ __forceinline__ void wait_loads_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
__device__ __forceinline__ void wait_loads_but8_barrier() {
  asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ---------------------------------------------------------------- kernel
// K step k (64 of K) reads A buffer k % 3 and W buffer k % 2 and is four
// substeps of 16 of K; a "phase" is the 16 MFMAs of one substep.  Each K step
// starts right after the barrier that published its tiles.  Its first phase
// runs the last substep of step k - 1 (fragments already in registers) beside
// the first fragment reads of step k; each later phase runs beside the next
// substep's fragment reads.  The 16 loads of a wave per K step are spread one
// per four MFMAs over all four phases: the W tile of step k + 1 in the first
// two (its buffer was last read in step k - 1), the A tile of step k + 2 in the
// last two (its buffer, (k - 1) % 3, too).  So the A loads have more than a K
// step to land, and no phase issues more than 16 loads per CU: the CU's
// address unit takes about 13 cycles per 16-byte load, and a burst of 64 (all
// of a K step's loads in one or two phases) stalls the waves that issue them.
// The barrier closing step k waits for all but this wave's 8 newest loads
// (step k + 2's A tile).  Every phase is a fixed sequence: sched_barrier keeps
// the compiler from regrouping it.
template <class Epi>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs a, Epi epi) {
  constexpr int BM = 256, BN = 256, TM = 128, TN = 128, FM = 4, FN = 4;
  constexpr uint32_t kNoRow = 0x80000000u;  // offset past every buffer range
  static_assert(2 * Epi::kSlotBytes(TN, TM) <= BM * BK * 2 * 2, "epilogue staging exceeds half the tile buffers");

  __shared__ __attribute__((aligned(1024))) bf16 sA[3][BM * BK];  // A ring: K step k in k % 3
  __shared__ __attribute__((aligned(1024))) bf16 sB[2][BN * BK];  // W ring: K step k in k % 2

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;

  const int tiles_m = cdiv(a.M, BM), tiles_n = epi.tiles_n(BN);
  const int lid = xcd_remap(blockIdx.x, gridDim.x);
  // Tile order: each die takes a contiguous range of tiles, swept in groups
  // of GM row tiles, column-major inside a group, so the tiles a die runs at
  // once share A and W panels in its L2.  When a row of tiles is at most 32
  // wide (the O and down projections: N = h), whole rows run at once (GM = 1):
  // every A panel is then read from HBM once and the small W is re-read from
  // the last-level cache.
  const int GM = tiles_n <= 32 ? 1 : 8;
  const int per_group = GM * tiles_n;
  const int first_m = (lid / per_group) * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int tm = first_m + (lid % per_group) % gsz;
  const int tn = (lid % per_group) / gsz;
  const int m0 = tm * BM;

  // Load q < 8 of wave w fills LDS chunks [(8w + q) 64, +64) of the A tile,
  // q >= 8 the same chunks of the W tile: lane l writes tile row
  // r = 8 (8w + q % 8) + l / 8 at swizzled chunk column l % 8, so it fetches
  // the logical chunk (l % 8) ^ ((r >> 1) & 7) of that row.  A's buffer starts
  // at the tile's first row and covers its valid rows; W rows an epilogue maps
  // to nothing get an offset past W's range, so rows outside the matrices read
  // as zero with no selects.  K advances in the scalar offset.
  const int rows_a = min(BM, a.M - m0);
  i32x4 ra, rw;
  {
    auto u = [](int x) { return __builtin_amdgcn_readfirstlane(x); };
    const uint64_t pa = (uint64_t)(a.A + (long)m0 * a.lda), pw = (uint64_t)a.W;
    ra = i32x4{u((int)pa), u((int)(pa >> 32)), u(rows_a * a.lda * 2), 0x00020000};
    rw = i32x4{u((int)pw), u((int)(pw >> 32)), u(a.w_bytes), 0x00020000};
  }
  uint32_t voff[16];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int r = 8 * (8 * wave + q) + (lane >> 3);
    const int kc = (lane & 7) ^ ((r >> 1) & 7);
    // rows r >= 8 (q % 4) hold at least (q % 4) KiB of offset (K >= 64), so
    // subtracting the group's instruction offset cannot wrap
    voff[q] = r < rows_a ? (uint32_t)(r * a.lda + kc * 8) * 2u - (q & 3) * 1024u : kNoRow;
    const int gr = epi.template w_row<BN, TN>(tn, r);
    voff[8 + q] = gr >= 0 ? (uint32_t)(gr * a.ldw + kc * 8) * 2u - (q & 3) * 1024u : kNoRow;
  }
  const uint32_t ldsA = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16*)&sA[0][0];
  const uint32_t ldsB = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16*)&sB[0][0];
  constexpr uint32_t kBuf = BM * BK * 2;  // bytes of one tile buffer
  // q < 8: A load into A buffer buf; q >= 8: W load into W buffer buf
  auto load = [&](int q, int buf, int k0) __attribute__((always_inline)) {
    const uint32_t lds = (q < 8 ? ldsA : ldsB) + buf * kBuf + (8 * wave + (q & 4)) * 1024;
    load_lds16(q < 8 ? ra : rw, voff[q], __builtin_amdgcn_readfirstlane(k0 * 2),
               __builtin_amdgcn_readfirstlane(lds), q & 3);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = zero16();

  // fragment f < 4: A block f, f >= 4: W block f - 4, of substep s of K step k
  bf16x8 fr[2][8];
  // a3 = k % 3 and b2 = k % 2: the ring slots of K step k's A and W tiles
  auto read_frag = [&](int a3, int b2, int s, int set, int f) __attribute__((always_inline)) {
    const int kci = s * 2 + (lane >> 5);
    if (f < 4)
      fr[set][f] = *reinterpret_cast<const bf16x8*>(&sA[a3][swz(wm * TM + f * 32 + (lane & 31), kci)]);
    else
      fr[set][f] = *reinterpret_cast<const bf16x8*>(&sB[b2][swz(wn * TN + (f - 4) * 32 + (lane & 31), kci)]);
  };
  // reads in the order the next phase's MFMAs need them
  constexpr int kReadOrder[8] = {0, 4, 5, 6, 7, 1, 2, 3};
  // One phase: the 16 MFMAs of the fragments in set mset (if MMA), the 8
  // fragment reads of substep rs of the K step in slots (a3, b2) into set rset
  // (if RD), one beside each of the first 8 MFMAs, and (if LD) 4 loads
  // q0 .. q0+3 of the K step at k0 into buffer dbuf, one per 4 MFMAs.  The
  // reads land during the phase's second half, so one wait at the head of the
  // next phase covers all of them (and the wait before the step's closing
  // barrier finds them done).
  auto phase = [&](auto MMA, auto RD, auto LD, int mset, int a3, int b2, int rs, int rset, int q0, int dbuf, int k0)
      __attribute__((always_inline)) {
    if constexpr (decltype(MMA)::value) __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      if constexpr (decltype(MMA)::value)
        acc[q >> 2][q & 3] = mfma_32x32x16(fr[mset][q >> 2], fr[mset][4 + (q & 3)], acc[q >> 2][q & 3]);
      if constexpr (decltype(RD)::value)
        if (q < 8) read_frag(a3, b2, rs, rset, kReadOrder[q]);
      if constexpr (decltype(LD)::value)
        if ((q & 3) == 0) load(q0 + (q >> 2), dbuf, k0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using T = std::true_type;
  using F = std::false_type;

  // K step k:
  //   phase 0: MFMAs of step k-1 substep 3, reads of step k substep 0,
  //            W loads 0-3 of step k+1
  //   phase 1: substep 0, reads of substep 1, W loads 4-7 of step k+1
  //   phase 2: substep 1, reads of substep 2, A loads 0-3 of step k+2
  //   phase 3: substep 2, reads of substep 3, A loads 4-7 of step k+2
  //   barrier: step k+1's W (this step) and A (previous step) have landed.
  // The prologue loads A and W of step 0 and A of step 1.
  const int ksteps = a.K / BK;
#pragma unroll
  for (int q = 0; q < 16; ++q) load(q, 0, 0);                       // A(0), W(0)
  if (ksteps > 1) {
#pragma unroll
    for (int q = 0; q < 8; ++q) load(q, 1, BK);                      // A(1)
    wait_loads_but8_barrier();
  } else {
    wait_loads_barrier();
  }
  // K step k, its ring slots a3 = k % 3, b2 = k % 2
  auto body = [&](int k, auto FIRST, auto LDW, auto LDA, int a3, int b2) __attribute__((always_inline)) {
    const int k1 = (k + 1) * BK, k2 = (k + 2) * BK;
    const int wb = 1 - b2, ab = a3 == 0 ? 2 : a3 - 1;   // (k + 1) % 2, (k + 2) % 3
    phase(std::integral_constant<bool, !decltype(FIRST)::value>{}, T{}, LDW, 1, a3, b2, 0, 0, 8, wb, k1);
    phase(T{}, T{}, LDW, 0, a3, b2, 1, 1, 12, wb, k1);
    phase(T{}, T{}, LDA, 1, a3, b2, 2, 0, 0, ab, k2);
    phase(T{}, T{}, LDA, 0, a3, b2, 3, 1, 4, ab, k2);
  };
  using B1 = std::true_type;
  using B0 = std::false_type;
  if (ksteps >= 3) {
    body(0, B1{}, T{}, T{}, 0, 0);
    wait_loads_but8_barrier();
    // K steps 1 .. ksteps-3, six per pass (the ring periods are 3 and 2), so
    // every LDS address of a step is a constant offset from a lane base: the
    // slot arithmetic (k % 3 by multiplication) had cost about 20 scalar
    // instructions at the head of every step, where they delay its second MFMA
    int k = 1;
    for (;;) {
#define BC_KSTEP(A3, B2)                \
      if (k + 2 >= ksteps) break;       \
      body(k, B0{}, T{}, T{}, A3, B2);  \
      wait_loads_but8_barrier();        \
      ++k;
      BC_KSTEP(1, 1) BC_KSTEP(2, 0) BC_KSTEP(0, 1) BC_KSTEP(1, 0) BC_KSTEP(2, 1) BC_KSTEP(0, 0)
#undef BC_KSTEP
    }
    body(ksteps - 2, B0{}, T{}, F{}, (ksteps - 2) % 3, (ksteps - 2) & 1);
    wait_loads_barrier();
    body(ksteps - 1, B0{}, F{}, F{}, (ksteps - 1) % 3, (ksteps - 1) & 1);
  } else if (ksteps == 2) {
    body(0, B1{}, T{}, F{}, 0, 0);
    wait_loads_barrier();
    body(1, B0{}, F{}, F{}, 1, 1);
  } else {
    body(0, B1{}, F{}, F{}, 0, 0);
  }
  phase(T{}, F{}, F{}, 1, 0, 0, 0, 0, 0, 0, 0);

  // every wave is past its last LDS read: the tile buffers become the
  // epilogue's staging area, 64 KiB (of the A ring, or the W ring) per pair of
  // waves
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  char* half = wave < 2 ? (char*)&sA[0][0] : (char*)&sB[0][0];
  epi.template apply<BN, TN, FM, FN>(acc, a.M, tn, m0 + wm * TM, wn, lane, half, wave & 1);
}

template <class Epi>
hipError_t launch(GemmArgs a, const Epi& epi, hipStream_t s) {
  const int tiles = cdiv(a.M, 256) * epi.tiles_n(256);
  if (tiles == 0) return hipSuccess;
  // operand offsets are 32-bit buffer offsets: W and a 256-row A panel must
  // stay below 2 GiB, and K must be whole 64-wide steps
  const long w_bytes = (long)epi.w_rows() * a.ldw * 2, a_panel = 256L * a.lda * 2;
  if (w_bytes >= (1L << 31) || a_panel >= (1L << 31) || a.K % BK || a.K <= 0) return hipErrorInvalidValue;
  a.w_bytes = (int)w_bytes;
  hipLaunchKernelGGL((gemm_kernel<Epi>), dim3(tiles), dim3(256), 0, s, a, epi);
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
