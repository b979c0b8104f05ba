// Sparse (integer-target) softmax cross-entropy over the first V of Vp
// logit columns (the loss of the data-parallel training step algorithm;
// appendix "Sparse Cross-Entropy Loss Forward / Backward").
//
// The fused kernel streams each logit row (Vp = 50,304 floats = 196.5 KiB,
// more than one CU's LDS) through registers exactly once: a 1024-thread
// block holds the row as float4 (<= 16 per thread), finds the row maximum,
// turns the row into exp2((z - max) log2 e) in place, sums it, and writes the
// gradient (p - onehot) * scale back over the logits.  No probability matrix
// is materialised; traffic is one read and one write of the logits.
#include "bt_internal.h"

namespace bt {
namespace {

constexpr float LOG2E_X = 1.4426950408889634f;
constexpr float LN2_X = 0.6931471805599453f;
constexpr int XT = 1024;  // threads per row

__device__ __forceinline__ float block_reduce(float v, float* red, bool is_max) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = is_max ? wave_max(v) : wave_sum(v);
  __syncthreads();  // red may still be read from a previous reduction
  if (lane == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
  for (int i = 1; i < XT / 64; ++i) r = is_max ? fmaxf(r, red[i]) : r + red[i];
  return r;
}

// MODE 0: forward only (loss_rows, lse).  MODE 1: fused (also dlogits in place).
template <int NPT, int MODE>
__global__ void __launch_bounds__(XT) xent_row_kernel(float* logits, const int32_t* __restrict__ targets,
                                                      float* __restrict__ loss_rows, float* __restrict__ lse_out,
                                                      float* dlogits, float scale, int V, int Vp) {
  __shared__ float red[XT / 64];
  __shared__ float s_zy;
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const int V4 = Vp >> 2;
  int y = targets[row];
  const bool bad = y < 0 || y >= V;
  if (bad) y = 0;
  const floatx4* zr = reinterpret_cast<const floatx4*>(logits + (long long)row * Vp);
  floatx4 z[NPT];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    const int c4 = tid + XT * i;
    // the fused pass reads and overwrites each logit exactly once: streaming
    // (non-temporal) accesses keep the 3.3 GB row stream out of the caches
    z[i] = c4 < V4 ? (MODE == 1 ? __builtin_nontemporal_load(zr + c4) : zr[c4])
                   : floatx4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (4 * c4 + k >= V) z[i][k] = -INFINITY;  // padded columns are outside the softmax
      if (4 * c4 + k == y) s_zy = z[i][k];       // the target logit, taken from registers: the
                                                 // row is overwritten in place below
      mx = fmaxf(mx, z[i][k]);
    }
  }
  mx = block_reduce(mx, red, true);  // its barriers also publish s_zy
  const float zy = s_zy;
  const float mxl = mx * LOG2E_X;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NPT; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      z[i][k] = exp2_hw(z[i][k] * LOG2E_X - mxl);
      s += z[i][k];
    }
  s = block_reduce(s, red, false);
  const float lse = mx + log2f(s) * LN2_X;
  if (tid == 0) {
    loss_rows[row] = bad ? NAN : lse - zy;
    lse_out[row] = lse;
  }
  if (MODE == 1) {
    const float inv = bad ? NAN : scale / s;  // an invalid target: NaN gradient row
    floatx4* dr = reinterpret_cast<floatx4*>(dlogits + (long long)row * Vp);
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int c4 = tid + XT * i;
      if (c4 < V4) {
        floatx4 o;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int c = 4 * c4 + k;
          o[k] = c < V ? z[i][k] * inv - (c == y ? scale : 0.f) : 0.f;
        }
        __builtin_nontemporal_store(o, dr + c4);
      }
    }
  }
}

// Fused pass for a 50,304-column class of rows (13 float4 per thread),
// persistent and pipelined: each block (one per CU; the prefetch buffer is
// most of the LDS) takes rows b, b + G, ...  While a row is reduced and
// written, the next row is already on its way: its first XS_PF float4 per
// thread are copied straight into LDS (global_load_lds, no registers) and
// the remaining XS_NR into a small register set.  The gradient stores go out
// as raw buffer stores, unconditionally (lanes past the row are dropped by
// the buffer's range check), so every wave issues exactly 13 of them per row
// and the wait for the prefetch at the next row can skip exactly those 13
// (the stores need not complete before the next row starts).  Measured on
// MI355X at 16384 x 50304 logits: 1.29 ms (5.1 TB/s) for the one-row-per-CU
// kernel below, 1.15 ms (5.7 TB/s) for this one.
constexpr int XS_NPT = 13, XS_PF = 9, XS_NR = XS_NPT - XS_PF;

// GRAD false: the forward alone (loss rows and lse; logits only read).
template <bool GRAD>
__global__ void __launch_bounds__(XT) xent_stream_kernel(float* logits, const int32_t* __restrict__ targets,
                                                         float* __restrict__ loss_rows, float* __restrict__ lse_out,
                                                         float scale, int M, int V, int Vp) {
  __shared__ __attribute__((aligned(16))) float pf[XS_PF * XT * 4];
  __shared__ float red[XT / 64];
  __shared__ float s_zy;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int V4 = Vp >> 2;
  const int G = gridDim.x;
  auto rsrc = [&](int row) {
    return __builtin_amdgcn_make_buffer_rsrc(logits + (long long)row * Vp, (short)0, Vp * 4, 0x00020000);
  };
  const unsigned voff = 16u * tid;  // byte offset of the thread's float4 in a 1024-float4 slice
  const unsigned lds_wave = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(__attribute__((address_space(3))) float*)pf + 1024u * wave);
  // prefetch of a row: the LDS part (every lane in range: V4 >= XS_PF XT) and the register part
  floatx4 nx[XS_NR];
  auto prefetch = [&](int row) {
    const float* zr = logits + (long long)row * Vp;
#pragma unroll
    for (int i = 0; i < XS_PF; ++i) copy16_to_lds_sbase(zr, voff + 16u * XT * i, lds_wave + 16u * XT * i);
    const auto r = rsrc(row);
#pragma unroll
    for (int j = 0; j < XS_NR; ++j)  // past the row: 0, masked below like the padded columns
      nx[j] = __builtin_amdgcn_raw_buffer_load_b128(r, voff, 16 * XT * (XS_PF + j), 2);
  };
  int row = blockIdx.x;
  if (row >= M) return;
  prefetch(row);
  wait_copies();
  for (; row < M; row += G) {
    // the prefetch of this row is complete once at most the 13 stores of the
    // previous row are outstanding; then every wave's part is visible
    if (GRAD)
      asm volatile("s_waitcnt vmcnt(13)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    floatx4 z[XS_NPT];
#pragma unroll
    for (int i = 0; i < XS_PF; ++i) z[i] = *reinterpret_cast<const floatx4*>(pf + 4 * (XT * i + tid));
#pragma unroll
    for (int j = 0; j < XS_NR; ++j) z[XS_PF + j] = nx[j];
    __syncthreads();  // every wave has read the buffer: it may be refilled
    if (row + G < M) prefetch(row + G);

    int y = targets[row];
    const bool bad = y < 0 || y >= V;
    if (bad) y = 0;
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < XS_NPT; ++i) {
      const int c4 = tid + XT * i;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (4 * c4 + k >= V) z[i][k] = -INFINITY;  // padded columns are outside the softmax
        if (4 * c4 + k == y) s_zy = z[i][k];       // the target logit, taken from registers: the
                                                   // row is overwritten in place below
        mx = fmaxf(mx, z[i][k]);
      }
    }
    mx = block_reduce(mx, red, true);  // its barriers also publish s_zy
    const float zy = s_zy;
    const float mxl = mx * LOG2E_X;
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < XS_NPT; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        z[i][k] = exp2_hw(z[i][k] * LOG2E_X - mxl);
        sum += z[i][k];
      }
    // its barriers also separate this row's reads of s_zy from the next row's write
    sum = block_reduce(sum, red, false);
    const float lse = mx + log2f(sum) * LN2_X;
    if (tid == 0) {
      loss_rows[row] = bad ? NAN : lse - zy;
      lse_out[row] = lse;
    }
    if (!GRAD) continue;
    const float inv = bad ? NAN : scale / sum;  // an invalid target: NaN gradient row
    const auto r = rsrc(row);
#pragma unroll
    for (int i = 0; i < XS_NPT; ++i) {
      const int c4 = tid + XT * i;
      floatx4 o;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int c = 4 * c4 + k;
        o[k] = c < V ? z[i][k] * inv - (c == y ? scale : 0.f) : 0.f;
      }
      __builtin_amdgcn_raw_buffer_store_b128(o, r, voff, 16 * XT * i, 2);  // non-temporal; past the row: dropped
    }
  }
}

// Backward from a stored lse, elementwise: each thread one group of XB_U
// float4 of a row (all loaded before any is written; no grid-stride loop),
// non-temporal.
constexpr int XB_U = 8;
__global__ void __launch_bounds__(256) xent_bwd_kernel(const float* logits, const float* __restrict__ lse,
                                                       const int32_t* __restrict__ targets, float* dlogits,
                                                       float scale, int V, int Vp) {
  const int V4 = Vp >> 2;
  const int nbx = (V4 + 256 * XB_U - 1) / (256 * XB_U);
  const int row = blockIdx.x / nbx, bx = blockIdx.x - row * nbx;
  const float l = lse[row] * LOG2E_X;
  const int y = targets[row];
  const float sc = (y < 0 || y >= V) ? NAN : scale;  // an invalid target: NaN gradient row
  const floatx4* zr = reinterpret_cast<const floatx4*>(logits + (long long)row * Vp);
  floatx4* dr = reinterpret_cast<floatx4*>(dlogits + (long long)row * Vp);
  const int c0 = bx * (256 * XB_U) + threadIdx.x;
  floatx4 z[XB_U];
#pragma unroll
  for (int u = 0; u < XB_U; ++u)
    if (c0 + 256 * u < V4) z[u] = __builtin_nontemporal_load(zr + c0 + 256 * u);
#pragma unroll
  for (int u = 0; u < XB_U; ++u) {
    const int c4 = c0 + 256 * u;
    if (c4 < V4) {
      floatx4 o;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int c = 4 * c4 + k;
        o[k] = c < V ? (exp2_hw(z[u][k] * LOG2E_X - l) - (c == y ? 1.f : 0.f)) * sc : 0.f;
      }
      __builtin_nontemporal_store(o, dr + c4);
    }
  }
}

bt_status xent_check(const void* logits, const void* targets, int M, int V, int Vp, const char* who) {
  BT_RETURN_IF(M < 0 || V < 1 || Vp < V || (Vp & 3), BT_ESHAPE,
               "%s: M=%d V=%d Vp=%d (need 1 <= V <= Vp, Vp multiple of 4)", who, M, V, Vp);
  BT_RETURN_IF(Vp > XT * 4 * 16, BT_ESHAPE, "%s: Vp=%d larger than %d is not supported", who, Vp, XT * 64);
  BT_RETURN_IF(M > 0 && (!logits || !targets), BT_EINVAL, "%s: NULL pointer", who);
  BT_RETURN_IF(logits && !aligned16(logits), BT_EALIGN, "%s: logits must be 16-byte aligned", who);
  return BT_OK;
}

// CUs of the current device (the streaming pass runs one block per CU).
int stream_cus() {
  static const int n = [] {
    int dev = 0, c = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    return c;
  }();
  return n;
}

template <int MODE>
bt_status launch_rows(float* logits, const int32_t* targets, float* loss_rows, float* lse, float* dlogits,
                      float scale, int M, int V, int Vp, hipStream_t s) {
  const int npt = (Vp / 4 + XT - 1) / XT;
  dim3 grid(M), block(XT);
#define BT_X(N) hipLaunchKernelGGL((xent_row_kernel<N, MODE>), grid, block, 0, s, logits, targets, loss_rows, lse, dlogits, scale, V, Vp)
  if (npt <= 1) BT_X(1);
  else if (npt <= 2) BT_X(2);
  else if (npt <= 4) BT_X(4);
  else if (npt <= 8) BT_X(8);
  else if (npt <= 13) BT_X(13);
  else BT_X(16);
#undef BT_X
  return check_launch("xent_row_kernel");
}

}  // namespace
}  // namespace bt

using namespace bt;

extern "C" bt_status bt_softmax_xent_fwd(const float* logits, const int32_t* targets, float* loss_rows, float* lse,
                                         int M, int V, int Vp, void* stream) {
  bt::clear_error();
  BT_TRY(xent_check(logits, targets, M, V, Vp, "bt_softmax_xent_fwd"));
  if (M == 0) return BT_OK;
  BT_RETURN_IF(!loss_rows || !lse, BT_EINVAL, "bt_softmax_xent_fwd: NULL output");
  const int V4 = Vp / 4;
  if (V4 > XT * (XS_NPT - 1) && V4 <= XT * XS_NPT) {
    const int cus = stream_cus();
    if (cus > 0) {
      hipLaunchKernelGGL(xent_stream_kernel<false>, dim3(M < cus ? M : cus), dim3(XT), 0, as_stream(stream),
                         const_cast<float*>(logits), targets, loss_rows, lse, 0.f, M, V, Vp);
      return check_launch("xent_stream_kernel");
    }
  }
  return launch_rows<0>(const_cast<float*>(logits), targets, loss_rows, lse, nullptr, 0.f, M, V, Vp,
                        as_stream(stream));
}

extern "C" bt_status bt_softmax_xent_bwd(const float* logits, const float* lse, const int32_t* targets,
                                         float* dlogits, float scale, int M, int V, int Vp, void* stream) {
  bt::clear_error();
  BT_TRY(xent_check(logits, targets, M, V, Vp, "bt_softmax_xent_bwd"));
  if (M == 0) return BT_OK;
  BT_RETURN_IF(!lse || !dlogits, BT_EINVAL, "bt_softmax_xent_bwd: NULL pointer");
  BT_RETURN_IF(!aligned16(dlogits), BT_EALIGN, "bt_softmax_xent_bwd: dlogits must be 16-byte aligned");
  const int V4 = Vp / 4;
  const long long nb = (long long)((V4 + 256 * XB_U - 1) / (256 * XB_U)) * M;
  BT_RETURN_IF(nb > 0x7fffffffLL, BT_ESHAPE, "bt_softmax_xent_bwd: M=%d too large", M);
  hipLaunchKernelGGL(xent_bwd_kernel, dim3((unsigned)nb), dim3(256), 0, as_stream(stream), logits, lse, targets,
                     dlogits, scale, V, Vp);
  return check_launch("xent_bwd_kernel");
}

extern "C" bt_status bt_softmax_xent_fused(float* logits, const int32_t* targets, float* loss_rows, float* lse,
                                           float scale, int M, int V, int Vp, void* stream) {
  bt::clear_error();
  BT_TRY(xent_check(logits, targets, M, V, Vp, "bt_softmax_xent_fused"));
  if (M == 0) return BT_OK;
  BT_RETURN_IF(!loss_rows || !lse, BT_EINVAL, "bt_softmax_xent_fused: NULL output");
  const int V4 = Vp / 4;
  if (V4 > XT * (XS_NPT - 1) && V4 <= XT * XS_NPT) {
    const int cus = stream_cus();
    if (cus > 0) {
      hipLaunchKernelGGL(xent_stream_kernel<true>, dim3(M < cus ? M : cus), dim3(XT), 0, as_stream(stream), logits,
                         targets, loss_rows, lse, scale, M, V, Vp);
      return check_launch("xent_stream_kernel");
    }
  }
  return launch_rows<1>(logits, targets, loss_rows, lse, logits, scale, M, V, Vp, as_stream(stream));
}
