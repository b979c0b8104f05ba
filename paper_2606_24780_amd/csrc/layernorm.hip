// LayerNorm forward and backward over the last dimension (pre-normalised
// GPT-2 blocks; appendix "LayerNorm Forward / Backward").
//
// One wave64 per row (up to four rows per wave in flight for short rows): the
// row (C <= 4096 floats) is held in registers as float4, mean and variance
// come from two in-register passes reduced with cross-lane shuffles (no LDS),
// so x is read once and y written once.  The
// backward computes dx row-wise the same way (two rows per wave in flight);
// dgamma/dbeta are accumulated per wave over a contiguous chunk of rows,
// combined per block through LDS and written as one partial row per block
// (at most 256 blocks), which a second kernel sums in a fixed order.
#include "bt_internal.h"

namespace bt {
namespace {

constexpr int ROWS_PER_BLOCK = 4;  // 4 waves

// Rows per wave of the forward: the fewer float4 a row takes per lane, the
// more rows a wave keeps in flight (4 for C <= 768, 2 for C <= 1024); four
// rows measured 10% faster than two at C = 768.
constexpr int ln_fwd_rpw(int nv) { return nv <= 3 ? 4 : (nv <= 4 ? 2 : 1); }

// RPW rows per wave (consecutive), all rows' loads issued before any row is
// reduced, so a wave keeps RPW rows of x in flight.
template <int NV, int RPW>
__global__ void __launch_bounds__(256) ln_fwd_kernel(const float* __restrict__ x,
                                                     const float* __restrict__ gamma,
                                                     const float* __restrict__ beta,
                                                     float* __restrict__ y, float* __restrict__ mean,
                                                     float* __restrict__ rstd, int M, int C, float eps) {
  const int lane = threadIdx.x & 63;
  const int row0 = (blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6)) * RPW;
  if (row0 >= M) return;
  const int C4 = C >> 2;
  floatx4 v[RPW][NV];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const floatx4* xr = reinterpret_cast<const floatx4*>(x + (long long)(row0 + r) * C);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane + 64 * i;
      v[r][i] = (c < C4 && row0 + r < M) ? xr[c] : floatx4{0.f, 0.f, 0.f, 0.f};
    }
  }
  const floatx4* g4 = reinterpret_cast<const floatx4*>(gamma);
  const floatx4* b4 = reinterpret_cast<const floatx4*>(beta);
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int row = row0 + r;
    if (row >= M) break;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) s += (v[r][i][0] + v[r][i][1]) + (v[r][i][2] + v[r][i][3]);
    const float mu = wave_sum(s) / (float)C;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane + 64 * i;
      if (c < C4) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float d = v[r][i][k] - mu;
          q += d * d;
        }
      }
    }
    const float var = wave_sum(q) / (float)C;
    const float rs = 1.0f / sqrtf(var + eps);
    floatx4* yr = reinterpret_cast<floatx4*>(y + (long long)row * C);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane + 64 * i;
      if (c < C4) {
        const floatx4 g = g4[c], b = b4[c];
        floatx4 o;
#pragma unroll
        for (int k = 0; k < 4; ++k) o[k] = (v[r][i][k] - mu) * rs * g[k] + b[k];
        yr[c] = o;
      }
    }
    if (lane == 0) {
      mean[row] = mu;
      rstd[row] = rs;
    }
  }
}

// Backward block: W waves (16 for rows up to 256 floats, fewer for wider
// rows so the registers suffice); each wave takes rows r0+w, r0+w+W, ... of
// the block's contiguous chunk, two rows at a time when they fit (both
// rows' loads issued before either row's reductions).
template <int NV>
struct BwdWaves {
  static constexpr int value = NV <= 1 ? 16 : (NV <= 4 ? 8 : 4);
};

template <int NV>
struct LnRow {
  floatx4 d[NV], xh[NV];  // dy and xhat of the row (g = dy * gamma is recomputed)
  floatx4 old[NV];        // dx before this call (accumulating calls), loaded with dy and x
  float mg, mgx, rs;
};

template <int NV>
__device__ __forceinline__ void ln_row_load(LnRow<NV>& r, const float* dy, const float* __restrict__ x,
                                            const float* __restrict__ mean, const float* __restrict__ rstd,
                                            const float* dx, bool accumulate, const floatx4 (&gam)[NV],
                                            int row, int C4, int lane) {
  const floatx4* dyr = reinterpret_cast<const floatx4*>(dy + (long long)row * 4 * C4);
  const floatx4* xr = reinterpret_cast<const floatx4*>(x + (long long)row * 4 * C4);
  const floatx4* dxr = reinterpret_cast<const floatx4*>(dx + (long long)row * 4 * C4);
  const float mu = mean[row];
  r.rs = rstd[row];
  floatx4 xv[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    r.d[i] = c < C4 ? dyr[c] : floatx4{0.f, 0.f, 0.f, 0.f};
    xv[i] = c < C4 ? __builtin_nontemporal_load(xr + c) : floatx4{0.f, 0.f, 0.f, 0.f};  // x: read once here
    r.old[i] = (accumulate && c < C4) ? dxr[c] : floatx4{0.f, 0.f, 0.f, 0.f};
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      r.xh[i][k] = c < C4 ? (xv[i][k] - mu) * r.rs : 0.f;
      const float g = r.d[i][k] * gam[i][k];
      s1 += g;
      s2 += g * r.xh[i][k];
    }
  }
  r.mg = s1;
  r.mgx = s2;
}

template <int NV>
__device__ __forceinline__ void ln_row_store(const LnRow<NV>& r, const floatx4 (&gam)[NV], float* dx, int row, int C4,
                                             int lane, float invC, float dx_beta, floatx4 (&acc_dg)[NV],
                                             floatx4 (&acc_db)[NV]) {
  const float mg = r.mg * invC, mgx = r.mgx * invC;
  floatx4* dxr = reinterpret_cast<floatx4*>(dx + (long long)row * 4 * C4);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    if (c < C4) {
      floatx4 o;
#pragma unroll
      for (int k = 0; k < 4; ++k) o[k] = r.rs * (r.d[i][k] * gam[i][k] - mg - r.xh[i][k] * mgx);
      if (dx_beta != 0.f) o += r.old[i];
      dxr[c] = o;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc_dg[i][k] += r.d[i][k] * r.xh[i][k];
        acc_db[i][k] += r.d[i][k];
      }
    }
  }
}

// dx row-wise; per-block partial column sums of dy*xhat and dy.
template <int NV, int BWD_WAVES = BwdWaves<NV>::value>
__global__ void __launch_bounds__(64 * BWD_WAVES) ln_bwd_kernel(const float* dy, const float* __restrict__ x,
                                                                const float* __restrict__ gamma,
                                                                const float* __restrict__ mean,
                                                                const float* __restrict__ rstd, float* dx,
                                                                float* __restrict__ part, int M, int C,
                                                                int rows_per_block, float dx_beta) {
  __shared__ floatx4 red[64 * NV][2];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int C4 = C >> 2;
  const float invC = 1.0f / (float)C;
  const floatx4* g4 = reinterpret_cast<const floatx4*>(gamma);
  floatx4 gam[NV], acc_dg[NV], acc_db[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    gam[i] = c < C4 ? g4[c] : floatx4{0.f, 0.f, 0.f, 0.f};
    acc_dg[i] = floatx4{0.f, 0.f, 0.f, 0.f};
    acc_db[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  const int r0 = blockIdx.x * rows_per_block;
  const int r1 = min(M, r0 + rows_per_block);
  const bool acc = dx_beta != 0.f;
  int row = r0 + wave;
  if (NV <= 4) {
    for (; row + BWD_WAVES < r1; row += 2 * BWD_WAVES) {
      LnRow<NV> a, b;
      ln_row_load<NV>(a, dy, x, mean, rstd, dx, acc, gam, row, C4, lane);
      ln_row_load<NV>(b, dy, x, mean, rstd, dx, acc, gam, row + BWD_WAVES, C4, lane);
      a.mg = wave_sum(a.mg);
      b.mg = wave_sum(b.mg);
      a.mgx = wave_sum(a.mgx);
      b.mgx = wave_sum(b.mgx);
      ln_row_store<NV>(a, gam, dx, row, C4, lane, invC, dx_beta, acc_dg, acc_db);
      ln_row_store<NV>(b, gam, dx, row + BWD_WAVES, C4, lane, invC, dx_beta, acc_dg, acc_db);
    }
  }
  for (; row < r1; row += BWD_WAVES) {
    LnRow<NV> a;
    ln_row_load<NV>(a, dy, x, mean, rstd, dx, acc, gam, row, C4, lane);
    a.mg = wave_sum(a.mg);
    a.mgx = wave_sum(a.mgx);
    ln_row_store<NV>(a, gam, dx, row, C4, lane, invC, dx_beta, acc_dg, acc_db);
  }
  // fixed-order combine of the waves (wave 0 first), one partial row per block
  for (int w = 0; w < BWD_WAVES; ++w) {
    if (wave == w) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int c = lane + 64 * i;
        if (w == 0) {
          red[c][0] = acc_dg[i];
          red[c][1] = acc_db[i];
        } else {
          red[c][0] += acc_dg[i];
          red[c][1] += acc_db[i];
        }
      }
    }
    __syncthreads();
  }
  floatx4* pg = reinterpret_cast<floatx4*>(part + (long long)blockIdx.x * 2 * C);
  for (int c = threadIdx.x; c < C4; c += 64 * BWD_WAVES) {
    pg[c] = red[c][0];
    pg[C4 + c] = red[c][1];
  }
}

int ln_nv(int C) { return (C / 4 + 63) / 64; }

// Waves per backward block for a row width (BwdWaves of the dispatched NV).
int ln_bwd_waves(int C) {
  const int nv = ln_nv(C);
  return nv <= 1 ? 16 : (nv <= 4 ? 8 : 4);
}

// Backward blocks: about two rows per wave (a block of W waves takes >= 2W
// rows), at most one block per CU so that few partial rows remain to be
// combined.  Short inputs (M = 2048 rows of the 2.42B model) still spread
// over every CU.
int ln_bwd_blocks(int M, int waves) {
  int nb = (M + 2 * waves - 1) / (2 * waves);
  if (nb > 256) nb = 256;
  if (nb < 1) nb = 1;
  return nb;
}

#define BT_LN_DISPATCH(NVV, ...)                       \
  switch (NVV) {                                       \
    case 1: __VA_ARGS__(1); break;                     \
    case 2: __VA_ARGS__(2); break;                     \
    case 3: __VA_ARGS__(3); break;                     \
    case 4: __VA_ARGS__(4); break;                     \
    case 5: case 6: __VA_ARGS__(6); break;             \
    case 7: case 8: __VA_ARGS__(8); break;             \
    case 9: case 10: case 11: case 12: __VA_ARGS__(12); break; \
    default: __VA_ARGS__(16); break;                   \
  }

bt_status ln_check(int M, int C, const char* who) {
  BT_RETURN_IF(M < 0 || C <= 0 || (C & 3) || C > 4096, BT_ESHAPE,
               "%s: C=%d must be a positive multiple of 4 <= 4096 (M=%d)", who, C, M);
  return BT_OK;
}

}  // namespace

int ln_bwd_partial_rows(int M, int C) { return M > 0 ? ln_bwd_blocks(M, ln_bwd_waves(C)) : 0; }

bt_status ln_bwd_rows(const float* dy, const float* x, const float* gamma, const float* mean, const float* rstd,
                      float* dx, float dx_beta, float* part, int M, int C, hipStream_t s) {
  BT_TRY(ln_check(M, C, "ln_bwd_rows"));
  if (M == 0) return BT_OK;
  const int nb = ln_bwd_partial_rows(M, C);
  const int rpb = (M + nb - 1) / nb;
#define BT_LN_BWD(NV) hipLaunchKernelGGL(ln_bwd_kernel<NV>, dim3(nb), dim3(64 * BwdWaves<NV>::value), 0, s, dy, x, gamma, mean, rstd, dx, part, M, C, rpb, dx_beta)
  BT_LN_DISPATCH(ln_nv(C), BT_LN_BWD)
#undef BT_LN_BWD
  return check_launch("ln_bwd_kernel");
}

}  // namespace bt

using namespace bt;

extern "C" bt_status bt_layernorm_fwd(const float* x, const float* gamma, const float* beta, float* y,
                                      float* mean, float* rstd, int M, int C, float eps, void* stream) {
  bt::clear_error();
  BT_TRY(ln_check(M, C, "bt_layernorm_fwd"));
  if (M == 0) return BT_OK;
  BT_RETURN_IF(!x || !gamma || !beta || !y || !mean || !rstd, BT_EINVAL, "bt_layernorm_fwd: NULL pointer");
  BT_RETURN_IF(!aligned16(x) || !aligned16(y) || !aligned16(gamma) || !aligned16(beta), BT_EALIGN,
               "bt_layernorm_fwd: x, y, gamma, beta must be 16-byte aligned");
  BT_RETURN_IF(x == y, BT_EINVAL, "bt_layernorm_fwd: y must not alias x");
  BT_RETURN_IF(!(eps >= 0.f), BT_EINVAL, "bt_layernorm_fwd: eps must be >= 0");
  const int rpw = ln_fwd_rpw(ln_nv(C));
  dim3 grid((M + ROWS_PER_BLOCK * rpw - 1) / (ROWS_PER_BLOCK * rpw));
  hipStream_t s = as_stream(stream);
#define BT_LN_FWD(NV) hipLaunchKernelGGL((ln_fwd_kernel<NV, ln_fwd_rpw(NV)>), grid, dim3(256), 0, s, x, gamma, beta, y, mean, rstd, M, C, eps)
  BT_LN_DISPATCH(ln_nv(C), BT_LN_FWD)
#undef BT_LN_FWD
  return check_launch("ln_fwd_kernel");
}

extern "C" size_t bt_layernorm_bwd_ws_bytes(int M, int C) {
  if (M <= 0 || C <= 0) return 0;
  return align_up((size_t)ln_bwd_blocks(M, ln_bwd_waves(C)) * 2 * C * sizeof(float), 256);
}

extern "C" bt_status bt_layernorm_bwd(const float* dy, const float* x, const float* gamma, const float* mean,
                                      const float* rstd, float* dx, float* dgamma, float* dbeta,
                                      float dx_beta, float param_beta, void* ws, size_t ws_bytes, int M,
                                      int C, void* stream) {
  bt::clear_error();
  BT_TRY(ln_check(M, C, "bt_layernorm_bwd"));
  BT_RETURN_IF((dx_beta != 0.f && dx_beta != 1.f) || (param_beta != 0.f && param_beta != 1.f), BT_EINVAL,
               "bt_layernorm_bwd: dx_beta and param_beta must be 0 or 1");
  BT_RETURN_IF(!dy || !x || !gamma || !mean || !rstd || !dx || !dgamma || !dbeta, BT_EINVAL,
               "bt_layernorm_bwd: NULL pointer");
  BT_RETURN_IF(!aligned16(dy) || !aligned16(x) || !aligned16(dx) || !aligned16(gamma), BT_EALIGN,
               "bt_layernorm_bwd: dy, x, dx, gamma must be 16-byte aligned");
  BT_RETURN_IF(dx == dy && dx_beta != 0.f, BT_EINVAL, "bt_layernorm_bwd: dx may alias dy only with dx_beta = 0");
  hipStream_t s = as_stream(stream);
  if (M == 0) {
    if (param_beta == 0.f) {
      BT_TRY(fill_zero(dgamma, (size_t)C, s));
      BT_TRY(fill_zero(dbeta, (size_t)C, s));
    }
    return BT_OK;
  }
  const size_t need = bt_layernorm_bwd_ws_bytes(M, C);
  BT_RETURN_IF(!ws || ws_bytes < need, BT_EWORKSPACE, "bt_layernorm_bwd: workspace of %zu bytes needed (got %zu)",
               need, ws_bytes);
  float* part = static_cast<float*>(ws);
  BT_TRY(ln_bwd_rows(dy, x, gamma, mean, rstd, dx, dx_beta, part, M, C, s));
  return sum_partials(part, ln_bwd_partial_rows(M, C), 2LL * C, 2 * C, dgamma, C, dbeta, param_beta, s);
}
