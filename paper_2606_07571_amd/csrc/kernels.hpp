// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on
// `stream` and returns the hipError_t of the launch.  Shapes are validated by
// the caller (runtime.cpp) before any launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

// ----- GEMM family: C = A[M,K] . W[N,K]^T, bf16 operands, fp32 accumulation.

// R[M, N] (fp32, row stride ldr) += A . W^T
hipError_t gemm_residual(const void* A, int lda, const void* W, int ldw, int M, int N, int K,
                         float* R, int ldr, hipStream_t s);

// act[M, F] (bf16) = silu(A . Wg^T) * (A . Wu^T), Wg = W rows [0, F), Wu = rows [F, 2F)
hipError_t gemm_swiglu(const void* A, int lda, const void* W, int ldw, int M, int F, int K,
                       void* act, hipStream_t s);

// Fused Q/K/V projection with rotate-half RoPE.  Row r of A is token
// t = r % n_seq of sequence b = r / n_seq at position pos0 + t.  Output column
// block j of W (head j, dh rows) goes to Q head j (j < Hq), K head j - Hq
// (j < Hq + Hkv) or V head j - Hq - Hkv; element (b, head, t, dim) of a part is
// stored at base + b*sb + head*sh + t*dh + dim (bf16).  The bias (bf16, one
// per output column, or null) is added first; Q and K are then rotated with
// the tables cos_t/sin_t [pos][dh/2].
struct QkvOut {
  void* q;
  void* k;
  void* v;
  long q_sb, q_sh, k_sb, k_sh, v_sb, v_sh;
  const void* bias = nullptr;
};
hipError_t gemm_qkv_rope(const void* A, int lda, const void* W, int ldw, int M, int K, int Hq,
                         int Hkv, int dh, int n_seq, int pos0, const float* cos_t,
                         const float* sin_t, const QkvOut& out, hipStream_t s);

// ----- attention: one launch of prefix + suffix bidirectional attention.
// Prefix K/V [Hkv][m][dh] (head stride p_sh elements, rows dh apart) are shared
// by every request when p_sb == 0; otherwise request b's prefix starts p_sb
// elements after request b-1's.  Suffix K/V are per request.  m may be 0
// (plain full attention of each request over its own n_s keys).
struct AttnArgs {
  const void* q;
  long q_sb, q_sh, q_sr;
  const void* kp;
  const void* vp;
  long p_sb, p_sh;
  const void* ks;
  const void* vs;
  long s_sb, s_sh, s_sr;
  void* out;
  long o_sb, o_sh, o_sr;
  int B, Hq, Hkv, m, n_s, dh;
  float scale;
  int out_f32;  // 1: fp32 output, 0: bf16 output
};
hipError_t attention(const AttnArgs& a, hipStream_t s);

// ----- KV similarity (Eq. 3): out[b * out_req + l * out_layer] =
// cos(flatten(a_l), flatten(r_{l,b})) for b < B, l < L.  Both sides are L
// layers x P parts x H heads x E contiguous elements (E a multiple of 8):
// cached element (l, p, g, i) at a + l*a_layer + p*a_part + g*a_head + i,
// request b's at r + l*r_layer + p*r_part + b*r_req + g*r_head + i (bf16).
// `partial` is scratch of kv_cosine_partial_bytes(v) bytes; out is fp64.
struct CosView {
  const void* a;
  long a_layer, a_part, a_head;
  const void* r;
  long r_layer, r_part, r_req, r_head;
  int L, P, H;
  long E;
  int B;
};
size_t kv_cosine_partial_bytes(const CosView& v);
// The allocation-free variant's scratch: cosine_scratch_bytes() bytes of
// device memory per GPU (a file-scope device array); *ptr = its address on the
// current device, looked up once per device; vectors of up to
// cosine_scratch_max_elements() elements fit.
size_t cosine_scratch_bytes();
long cosine_scratch_max_elements();
hipError_t cosine_scratch(double** ptr);
hipError_t kv_cosine(const CosView& v, double* partial, double* out, long out_req, long out_layer,
                     hipStream_t s);

// ----- deep-store header: 8 words a refresh step writes after the store's
// K/V blocks and a reuse step checks (see runtime.cpp)
struct DeepHeader {
  uint64_t w[8];
};
// hdr[0..8) = h.w (device, 8-byte aligned)
hipError_t deep_header_write(uint64_t* hdr, const DeepHeader& h, hipStream_t s);
// if hdr[0..8) differs from h.w anywhere, out[0..n) = NaN; otherwise nothing
hipError_t deep_header_check(const uint64_t* hdr, const DeepHeader& h, float* out, long n,
                             hipStream_t s);

// ----- elementwise / normalisation
// out[r, :] = bf16(x[r, :] / sqrt(mean(x[r, :]^2) + eps) * gain)
hipError_t rmsnorm(const float* x, const void* gain, void* out, int rows, int h, float eps,
                   hipStream_t s);
// out[i] = float(in[i])
hipError_t bf16_to_f32(const void* in, float* out, long n, hipStream_t s);
// R[b, t, :] = t < m ? pre[t, :] : suf[b, t - m, :]   (all fp32, row length h)
hipError_t build_full_residual(const float* pre, const float* suf, float* R, int B, int m,
                               int n_s, int h, hipStream_t s);
// out[b, t, :] = R[b, m + t, :]
hipError_t gather_suffix(const float* R, float* out, int B, int m, int n_s, int h,
                         hipStream_t s);
// cos_t/sin_t[p, i] = cos/sin(p * theta^(-2i/dh)), p in [0, n_pos), i in [0, dh/2)
hipError_t rope_table(float* cos_t, float* sin_t, int n_pos, int dh, double theta,
                      hipStream_t s);

}  // namespace bc
