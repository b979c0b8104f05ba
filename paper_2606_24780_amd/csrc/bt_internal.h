// Internal helpers shared by the libbt translation units (HIP, gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstddef>
#include <cstdint>
#include <cstdio>

#include "../../include/bt.h"

namespace bt {

// Thread-local error detail; set_error returns the status so call sites can
// `return fail(BT_ESHAPE, "...")`.
bt_status fail(bt_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// After a launch: turn a launch error into BT_EHIP.
bt_status check_launch(const char* what);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Zero n floats with a small kernel (no memset node).
bt_status fill_zero(float* p, size_t n, hipStream_t s);

// Fixed-order sum of per-block partial rows: for c < n,
//   dst[c] = beta * dst[c] + sum_{b < nb} part[b * ld + c],
// where dst is out_a[c] for c < n_a and out_b[c - n_a] otherwise.
bt_status sum_partials(const float* part, int nb, long long ld, int n, float* out_a, int n_a, float* out_b,
                       float beta, hipStream_t s);

// Several independent sums of the shape above (same nb, ld, n, n_a, beta),
// one per set, in as few launches as the kernel-argument budget allows
// (each set's result is bitwise that of sum_partials).
struct PartialSet {
  const float* part;
  float* out_a;
  float* out_b;
};
bt_status sum_partials_batched(const PartialSet* sets /*host*/, int nsets, int nb, long long ld, int n, int n_a,
                               float beta, hipStream_t s);

// Row pass of the LayerNorm backward alone: dx exactly as bt_layernorm_bwd
// (dx_beta 0 or 1), and one partial row of the dgamma (first C) / dbeta
// (next C) column sums per block in part[ln_bwd_partial_rows(M, C)][2 C],
// to be combined by sum_partials(part, nb, 2C, 2C, dgamma, C, dbeta, ...).
int ln_bwd_partial_rows(int M, int C);
bt_status ln_bwd_rows(const float* dy, const float* x, const float* gamma, const float* mean, const float* rstd,
                      float* dx, float dx_beta, float* part, int M, int C, hipStream_t s);

// Batch of products C_y = A_y B_y (A [M][K] row-major, B [K][N] row-major),
// batch y < nb nh at A + (y / nh) sa_b + (y % nh) sa_h (likewise B, C), in
// which output rows of each 128-row tile starting at m0 sum only k < m0 + 128
// (exact when A_y[m][k] = 0 for k > m, e.g. causal attention scores).
bt_status gemm_causal_batched(int M, int N, int K, const float* A, int lda, long long sa_b, long long sa_h,
                              const float* B, int ldb, long long sb_b, long long sb_h, float* C, int ldc,
                              long long sc_b, long long sc_h, int nb, int nh, hipStream_t stream);
// Segmented variant (context-parallel attention): rows of A and C are 1 or 2
// segments of `seg` rows at positions q_pos[], the K range 1 or 2 segments at
// k_pos[] (seg and positions multiples of 128); row tile sums the k whose
// positions do not exceed its last row's.  C = product + beta C, beta 0 or 1.
bt_status gemm_segmented_batched(int M, int N, int K, const float* A, int lda, long long sa_b, long long sa_h,
                                 const float* B, int ldb, long long sb_b, long long sb_h, float* C, int ldc,
                                 long long sc_b, long long sc_h, int nb, int nh, float beta, int seg,
                                 const int* q_pos, const int* k_pos, hipStream_t stream);

// Embedding backward buffers of the composed step: the token index
// (bt_embedding_index) and the backward's run partials.
size_t emb_index_bytes(long long M);
size_t emb_bwd_partials_bytes(long long M, int C);

// ------------------------------------------------------------------ device
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Direct global -> LDS copy of 16 bytes per lane (gfx950 global_load_lds_dwordx4):
// lane L of the wave writes LDS bytes [dst + 16 L, dst + 16 L + 16), dst
// wave-uniform, passed in M0.  The data never occupies VGPRs and needs no
// LDS store instruction.  It is issued from inline assembly so that the
// compiler does not conservatively wait for it before unrelated LDS reads
// of the other buffer; completion is awaited explicitly (wait_copies) before
// the barrier that publishes the tile.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void copy16_to_lds(const float* src, float* lds_dst) {
  const unsigned l = (unsigned)(uintptr_t)(__attribute__((address_space(3))) float*)lds_dst;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(l)), "v"(src)
               : "memory", "m0");
}
// The same copy with a wave-uniform global base (SGPR pair), a per-lane
// 32-bit byte offset and a wave-uniform LDS byte address.
__device__ __forceinline__ void copy16_to_lds_sbase(const float* base, unsigned voff, unsigned lds_byte) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds_byte), "v"(voff), "s"(base)
               : "memory", "m0");
}
#pragma clang diagnostic pop
__device__ __forceinline__ void wait_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// 2^x as the single hardware transcendental (v_exp_f32, about 1 ulp),
// without the library's rescaling for results below 2^-126: those may come
// out as 0, an absolute error under 1.2e-38.  Used where the exponent is a
// softmax logit minus its running maximum, so every result is in [0, 1].
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// tanh-form GELU and its derivative (FP32), evaluated through the logistic
// function: 1 + tanh(u) = 2 s with s = 1 / (1 + exp(-2u)), so
//   gelu(x)  = x s
//   gelu'(x) = s + 2 x s (1 - s) u'(x),   u = sqrt(2/pi) (x + 0.044715 x^3).
// Both s and 1 - s are formed without cancellation (the exponent is always
// <= 0), which keeps the tails accurate where 1 +- tanh(u) would round away.
// The exponential and the reciprocal are the single hardware instructions
// (v_exp_f32 on the base-2 exponent, v_rcp_f32; about 1 ulp each): this runs
// in GEMM epilogues over every element of the MLP activations, where the
// library expf and an IEEE division cost ~40 instructions per element.
// e underflowing to 0 (|u| > 43) changes s or 1 - s by less than 1e-37.
__device__ __forceinline__ void gelu_logistic(float x, float& s, float& oms, float& du) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float k1 = 0.044715f;
  const float m2log2e = -2.0f * 1.4426950408889634f;
  const float x2 = x * x;
  const float u = k0 * (x + k1 * x2 * x);
  du = k0 * (1.0f + 3.0f * k1 * x2);
  const float e = exp2_hw(m2log2e * fabsf(u));  // exp(-2|u|), in [0, 1]
  const float r = __builtin_amdgcn_rcpf(1.0f + e);
  if (u >= 0.f) {
    s = r;
    oms = e * r;
  } else {
    s = e * r;
    oms = r;
  }
}

__device__ __forceinline__ float gelu_f(float x) {
  float s, oms, du;
  gelu_logistic(x, s, oms, du);
  return x * s;
}

__device__ __forceinline__ float gelu_grad_f(float x) {
  float s, oms, du;
  gelu_logistic(x, s, oms, du);
  return s + 2.0f * x * s * oms * du;
}

}  // namespace bt

#define BT_CHECK_HIP(expr)                                                          \
  do {                                                                              \
    hipError_t _e = (expr);                                                         \
    if (_e != hipSuccess)                                                           \
      return ::bt::fail(BT_EHIP, "%s: %s", #expr, hipGetErrorString(_e));           \
  } while (0)

#define BT_RETURN_IF(cond, status, ...)                                             \
  do {                                                                              \
    if (cond) return ::bt::fail(status, __VA_ARGS__);                               \
  } while (0)

#define BT_TRY(expr)                                                                \
  do {                                                                              \
    bt_status _s = (expr);                                                          \
    if (_s != BT_OK) return _s;                                                     \
  } while (0)
