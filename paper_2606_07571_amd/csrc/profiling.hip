// KV similarity of Eq. 3 on gfx950: sim = cos(flatten(KV$_l), flatten(KV^ref))
// for every request of a batch, as an HBM-bound reduction.
//
// Both operands are P parts (K, V) x H heads x E contiguous elements (one
// head's prefix rows, E = m * dh).  The cached side is the same for every
// request: a workgroup takes one 8192-element chunk of one (part, head), reads
// the cached elements once and the same elements of up to 16 requests'
// reference copies, and accumulates per lane, in fp32, the squared norm of the
// cached chunk and per request the dot product and the reference's squared
// norm (each lane adds 32 products, so fp32 loses nothing that matters).  The
// workgroup reduces them in fp64 and stores its partial sums; a second kernel
// adds the partials of every workgroup in a fixed order in fp64 and writes
// dot / sqrt(|a|^2 |b|^2).  No atomics: results repeat bit for bit.
//
// Loads are 16 bytes per lane with consecutive lanes on consecutive
// addresses; the cached chunk is read once per 16 requests, so the bytes
// moved are (1/16 + 1) x the reference copies, the reduction's floor.
#include "device_common.hpp"
#include "kernels.hpp"

namespace bc {
namespace {

constexpr int kThreads = 256;
constexpr int kVecs = 4;                            // 16-byte vectors per lane per chunk
constexpr long kChunk = (long)kThreads * kVecs * 8;  // elements per workgroup
constexpr int kMaxReq = 16;                          // requests per pass
constexpr int kVals = 1 + 2 * kMaxReq;               // |a|^2, then dot and |r|^2 per request

__host__ __device__ constexpr long cdivl(long a, long b) { return (a + b - 1) / b; }

__device__ __forceinline__ void widen8(const u32x4& w, float (&f)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Sum of `v` over the workgroup in fp64, in a fixed order; every thread gets it.
__device__ double block_sum(double v, double* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int w = 0; w < kThreads / kWave; ++w) t += red[w];
  return t;
}

// grid.x: chunks per (part, head); grid.y: P * H.  Requests b0 .. b0 + nb - 1.
__global__ void __launch_bounds__(kThreads) cos_partial_kernel(CosView v, int b0, int nb,
                                                               double* __restrict__ partial) {
  __shared__ double red[kThreads / kWave];
  const int ph = blockIdx.y, p = ph / v.H, g = ph % v.H;
  const long base = (long)blockIdx.x * kChunk;
  const bf16* a = (const bf16*)v.a + p * v.a_part + g * v.a_head;
  const bf16* r = (const bf16*)v.r + p * v.r_part + (long)b0 * v.r_req + g * v.r_head;

  float na = 0.f;
  float dot[kMaxReq], nr[kMaxReq];
#pragma unroll
  for (int j = 0; j < kMaxReq; ++j) dot[j] = nr[j] = 0.f;
#pragma unroll
  for (int k = 0; k < kVecs; ++k) {
    const long i = base + ((long)k * kThreads + threadIdx.x) * 8;
    if (i >= v.E) break;
    float fa[8];
    widen8(*reinterpret_cast<const u32x4*>(a + i), fa);
#pragma unroll
    for (int e = 0; e < 8; ++e) na = fmaf(fa[e], fa[e], na);
#pragma unroll
    for (int j = 0; j < kMaxReq; ++j) {
      if (j < nb) {
        float fr[8];
        widen8(*reinterpret_cast<const u32x4*>(r + j * v.r_req + i), fr);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          dot[j] = fmaf(fa[e], fr[e], dot[j]);
          nr[j] = fmaf(fr[e], fr[e], nr[j]);
        }
      }
    }
  }
  double* out = partial + ((long)blockIdx.y * gridDim.x + blockIdx.x) * kVals;
  const double s_na = block_sum((double)na, red);
  if (threadIdx.x == 0) out[0] = s_na;
  for (int j = 0; j < nb; ++j) {
    const double s_dot = block_sum((double)dot[j], red);
    const double s_nr = block_sum((double)nr[j], red);
    if (threadIdx.x == 0) {
      out[1 + 2 * j] = s_dot;
      out[2 + 2 * j] = s_nr;
    }
  }
}

// One workgroup per request of the pass: the fixed-order fp64 sum of every
// workgroup's partials, then the cosine.
__global__ void __launch_bounds__(kThreads) cos_final_kernel(const double* __restrict__ partial,
                                                             long n_blocks, int b0, double* out,
                                                             long out_stride) {
  __shared__ double red[kThreads / kWave];
  const int j = blockIdx.x;
  double na = 0.0, dot = 0.0, nr = 0.0;
  for (long q = threadIdx.x; q < n_blocks; q += kThreads) {
    const double* pq = partial + q * kVals;
    na += pq[0];
    dot += pq[1 + 2 * j];
    nr += pq[2 + 2 * j];
  }
  na = block_sum(na, red);
  dot = block_sum(dot, red);
  nr = block_sum(nr, red);
  if (threadIdx.x == 0) out[(long)(b0 + j) * out_stride] = dot / sqrt(na * nr);
}

}  // namespace

size_t kv_cosine_partial_bytes(const CosView& v) {
  const long n_blocks = cdivl(v.E, kChunk) * v.P * v.H;
  return (size_t)n_blocks * kVals * sizeof(double);
}

hipError_t kv_cosine(const CosView& v, double* partial, double* out, long out_stride, hipStream_t s) {
  if (v.E <= 0 || v.E % 8 || v.P < 1 || v.H < 1 || v.B < 1) return hipErrorInvalidValue;
  const long chunks = cdivl(v.E, kChunk);
  if (chunks > INT32_MAX || (long)v.P * v.H > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)chunks, (unsigned)(v.P * v.H));
  for (int b0 = 0; b0 < v.B; b0 += kMaxReq) {
    const int nb = v.B - b0 < kMaxReq ? v.B - b0 : kMaxReq;
    hipLaunchKernelGGL(cos_partial_kernel, grid, dim3(kThreads), 0, s, v, b0, nb, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(cos_final_kernel, dim3(nb), dim3(kThreads), 0, s, partial,
                       chunks * v.P * v.H, b0, out, out_stride);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace bc
