// KV similarity of Eq. 3 on gfx950: sim = cos(flatten(KV$_l), flatten(KV^ref))
// for every request of a batch and every layer, as an HBM-bound reduction.
//
// Both operands are L layers x P parts (K, V) x H heads x E contiguous
// elements (one head's prefix rows, E = m * dh).  The cached side is the same
// for every request: a workgroup takes one 8192-element chunk of one (layer,
// part, head), reads the cached elements once and the same elements of up to
// 16 requests' reference copies, and accumulates per lane, in fp32, the
// squared norm of the cached chunk and per request the dot product and the
// reference's squared norm (each lane adds 32 products, so fp32 loses nothing
// that matters).  The lane sums go through LDS and are added per value in
// fp64 in a fixed order, giving the workgroup's partial sums; a second kernel
// adds the partials of every workgroup of a (layer, request) in a fixed order
// in fp64 and writes dot / sqrt(|a|^2 |b|^2).  No atomics: results repeat bit
// for bit, and a request's result does not depend on the others in its batch.
//
// Loads are 16 bytes per lane with consecutive lanes on consecutive
// addresses, non-temporal (every byte is read once), issued four requests at
// a time ahead of the arithmetic that consumes them; the cached chunk is read
// once per 16 requests, so the bytes moved are (1/16 + 1) x the reference
// copies, the reduction's floor.  Every layer goes in one launch.
#include <mutex>

#include "device_common.hpp"
#include "kernels.hpp"

namespace bc {
namespace {

constexpr int kThreads = 256;
constexpr int kVecs = 4;                            // 16-byte vectors per lane per chunk
constexpr long kChunk = (long)kThreads * kVecs * 8;  // elements per workgroup
constexpr int kMaxReq = 16;                          // requests per pass
constexpr int kGroup = 4;                            // requests whose loads are issued together
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

// grid.x: chunks per (layer, part, head); grid.y: L * P * H.  Requests
// b0 .. b0 + nb - 1.  Vector k of a lane covers elements
// base + (k * kThreads + tid) * 8 .. + 7 of its (layer, part, head).
__global__ void __launch_bounds__(kThreads) cos_partial_kernel(CosView v, int b0, int nb,
                                                               double* __restrict__ partial) {
  __shared__ float lsum[kVals][kThreads];
  const int lph = blockIdx.y, ph = lph % (v.P * v.H), l = lph / (v.P * v.H);
  const int p = ph / v.H, g = ph % v.H;
  const long base = (long)blockIdx.x * kChunk;
  const bf16* a = (const bf16*)v.a + l * v.a_layer + p * v.a_part + g * v.a_head;
  const bf16* r = (const bf16*)v.r + l * v.r_layer + p * v.r_part + (long)b0 * v.r_req + g * v.r_head;
  const int tid = threadIdx.x;
  int nk = 0;   // vectors of this lane inside the E elements
#pragma unroll
  for (int k = 0; k < kVecs; ++k)
    if (base + ((long)k * kThreads + tid) * 8 < v.E) nk = k + 1;

  u32x4 av[kVecs];
#pragma unroll
  for (int k = 0; k < kVecs; ++k)
    if (k < nk) av[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a + base + ((long)k * kThreads + tid) * 8));
  float na = 0.f;
#pragma unroll
  for (int k = 0; k < kVecs; ++k) {
    if (k < nk) {
      float fa[8];
      widen8(av[k], fa);
#pragma unroll
      for (int e = 0; e < 8; ++e) na = fmaf(fa[e], fa[e], na);
    }
  }
  lsum[0][tid] = na;
#pragma unroll
  for (int j0 = 0; j0 < kMaxReq; j0 += kGroup) {
    if (j0 >= nb) break;
    u32x4 rv[kGroup][kVecs];
#pragma unroll
    for (int jj = 0; jj < kGroup; ++jj)
#pragma unroll
      for (int k = 0; k < kVecs; ++k)
        if (j0 + jj < nb && k < nk)
          rv[jj][k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
              r + (j0 + jj) * v.r_req + base + ((long)k * kThreads + tid) * 8));
#pragma unroll
    for (int jj = 0; jj < kGroup; ++jj) {
      if (j0 + jj >= nb) break;
      float dot = 0.f, nr = 0.f;
#pragma unroll
      for (int k = 0; k < kVecs; ++k) {
        if (k < nk) {
          float fa[8], fr[8];
          widen8(av[k], fa);
          widen8(rv[jj][k], fr);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            dot = fmaf(fa[e], fr[e], dot);
            nr = fmaf(fr[e], fr[e], nr);
          }
        }
      }
      lsum[1 + 2 * (j0 + jj)][tid] = dot;
      lsum[2 + 2 * (j0 + jj)][tid] = nr;
    }
  }
  __syncthreads();
  // value q is added by wave q % 4: lane i sums lanes i, i+64, i+128, i+192 in
  // fp64, then the wave's fixed xor tree
  const int wave = tid >> 6, lane = tid & 63;
  double* out = partial + ((long)blockIdx.y * gridDim.x + blockIdx.x) * kVals;
  for (int q = wave; q < 1 + 2 * nb; q += kThreads / kWave) {
    double t = (double)lsum[q][lane];
#pragma unroll
    for (int i = 1; i < kThreads / kWave; ++i) t += (double)lsum[q][lane + 64 * i];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o, kWave);
    if (lane == 0) out[q] = t;
  }
}

// One workgroup per (request of the pass, layer): the fixed-order fp64 sum of
// the partials of the layer's workgroups, then the cosine.
__global__ void __launch_bounds__(kThreads) cos_final_kernel(const double* __restrict__ partial,
                                                             long blocks_per_layer, int b0,
                                                             double* out, long out_req,
                                                             long out_layer) {
  __shared__ double red[kThreads / kWave];
  const int j = blockIdx.x, l = blockIdx.y;
  const double* pl = partial + (long)l * blocks_per_layer * kVals;
  double na = 0.0, dot = 0.0, nr = 0.0;
  for (long q = threadIdx.x; q < blocks_per_layer; q += kThreads) {
    const double* pq = pl + q * kVals;
    na += pq[0];
    dot += pq[1 + 2 * j];
    nr += pq[2 + 2 * j];
  }
  na = block_sum(na, red);
  dot = block_sum(dot, red);
  nr = block_sum(nr, red);
  if (threadIdx.x == 0) out[(long)(b0 + j) * out_req + (long)l * out_layer] = dot / sqrt(na * nr);
}

}  // namespace

// Scratch of the allocation-free cosine (bc_cosine_similarity_noalloc): the
// per-workgroup partial sums of one reduction live in this file-scope device
// array instead of a caller's workspace.  Every GPU the library runs on holds
// its own copy until the process ends; every call on a GPU shares it.  Each
// partial is written before it is read, so nothing needs clearing between
// calls; calls that overlap on one GPU race on it.
constexpr size_t kCosScratchBytes = 4u << 20;
static __device__ __align__(256) double scratch[kCosScratchBytes / sizeof(double)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

size_t cosine_scratch_bytes() { return kCosScratchBytes; }

long cosine_scratch_max_elements() {
  return (long)(kCosScratchBytes / (kVals * sizeof(double))) * kChunk;
}

hipError_t cosine_scratch(double** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    // the array's name is a host-side stand-in: only the address the runtime
    // reports for the current device may reach a kernel
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = static_cast<double*>(p);
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

size_t kv_cosine_partial_bytes(const CosView& v) {
  const long n_blocks = cdivl(v.E, kChunk) * v.P * v.H * v.L;
  return (size_t)n_blocks * kVals * sizeof(double);
}

hipError_t kv_cosine(const CosView& v, double* partial, double* out, long out_req, long out_layer,
                     hipStream_t s) {
  if (v.E <= 0 || v.E % 8 || v.P < 1 || v.H < 1 || v.B < 1 || v.L < 1) return hipErrorInvalidValue;
  const long chunks = cdivl(v.E, kChunk);
  if (chunks > INT32_MAX || (long)v.L * v.P * v.H > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)chunks, (unsigned)(v.L * v.P * v.H));
  for (int b0 = 0; b0 < v.B; b0 += kMaxReq) {
    const int nb = v.B - b0 < kMaxReq ? v.B - b0 : kMaxReq;
    hipLaunchKernelGGL(cos_partial_kernel, grid, dim3(kThreads), 0, s, v, b0, nb, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(cos_final_kernel, dim3(nb, v.L), dim3(kThreads), 0, s, partial,
                       chunks * v.P * v.H, b0, out, out_req, out_layer);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace bc
