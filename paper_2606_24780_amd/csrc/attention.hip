// Causal multi-head attention, forward and backward, FP32 on the CDNA4
// matrix cores (v_mfma_f32_32x32x2_f32), tiled with an online softmax so the
// T x T score matrix never reaches HBM.
//
// Problem (GPT-2 architecture figure: masked multi-head self-attention;
// appendix "Attention Forward/Backward", causal case): per batch b and head h,
//   S = Q K^T / sqrt(hd),  key j visible to query i iff j <= i,
//   P = softmax(S),  O = P V,  lse_i = log sum_j exp(S_ij).
// Backward, with D_i = sum_d dO_id O_id:
//   dV = P^T dO,  dP = dO V^T,  dS = P o (dP - D),  dQ = dS K / sqrt(hd),
//   dK = dS^T Q / sqrt(hd).
//
// Layout: qkv [B, T, 3, H, hd] (the QKV projection output), out [B, T, H, hd],
// lse [B, H, T], dqkv like qkv.
//
// Design (gfx950, wave64):
//  * a block = 4 waves = 128 query rows (forward, dQ) or 128 key rows (dK/dV);
//    each wave owns 32 rows and keeps its row operand (Q, or K and V) in
//    registers; the streamed operand tiles of 32 rows are double-buffered in
//    LDS and shared by the 4 waves.
//  * products are computed transposed where that makes the next product's
//    operand a register the lane already holds: S^T = K Q^T leaves each lane
//    with one query's 16 scores, so the softmax row statistics are in-lane plus
//    one exchange with lane^32, and the probabilities are directly the B
//    operand of O^T += V^T P^T (k-slot of register r: row 8(r/4) + 4 h + r%4).
//  * exp is computed as exp2 with log2(e)/sqrt(hd) folded into the register
//    operand.
//  * backward is deterministic (no atomics).  With the full workspace:
//    D = rowsum(dO o O) in a small kernel, then one key-major kernel
//    recomputes P from lse, accumulates dK and dV and also writes dS / sqrt(hd)
//    to the workspace (B H T T floats), and dQ = dS K is one batched product
//    on the GEMM kernel (causal: each 128-row tile sums only keys below its
//    end).  This drops the second recomputation of S and dP that a separate
//    query-major dQ kernel needs.  With only the small workspace, a query-major
//    kernel (D, dQ) recomputes S and dP instead (no T^2 memory).
//  * causal blocks above the diagonal are skipped per wave; blocks are
//    launched heaviest first.
//  * head dims up to 128 (multiple of 4), zero-padded to 32, 64 or 128
//    inside the kernels; at 128 the key-major backward keeps its dK/dV
//    accumulators partly in AGPRs at one wave per SIMD.
#include "bt_internal.h"

namespace bt {
namespace {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

__device__ __forceinline__ floatx16 mfma32(float a, float b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ void zero16(floatx16& v) {
#pragma unroll
  for (int r = 0; r < 16; ++r) v[r] = 0.f;
}

// accumulator row (within a 32 x 32 block) of register r for lane half hh
__device__ __forceinline__ int acc_row(int r, int hh) { return 8 * (r >> 2) + 4 * hh + (r & 3); }

struct AttnShape {
  int B, T, H, hd;
  long long row_stride;  // floats between consecutive tokens in qkv (3 H hd)
};

// Load rows [r0, r0 + 32) of one of Q/K/V/dO-like matrices into an LDS tile
// [32][LD] (zero-filled beyond T or hd). src points at (b, token 0, head h);
// `stride` is the token stride.  256 threads, HDP/4 float4 per row.
template <int HDP, int LD>
__device__ __forceinline__ void load_rows(floatx4 (&r)[HDP / 32], const float* __restrict__ src,
                                          long long stride, int r0, int T, int hd, int tid) {
  constexpr int PER_ROW = HDP / 4;            // float4 per row
  constexpr int ROWS_PER_PASS = 256 / PER_ROW;
#pragma unroll
  for (int i = 0; i < HDP / 32; ++i) {
    const int row = tid / PER_ROW + ROWS_PER_PASS * i;
    const int d = 4 * (tid % PER_ROW);
    const int t = r0 + row;
    if (t < T && d < hd)
      r[i] = *reinterpret_cast<const floatx4*>(src + (long long)t * stride + d);
    else
      r[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
}

template <int HDP, int LD>
__device__ __forceinline__ void store_rows(float* __restrict__ s, const floatx4 (&r)[HDP / 32], int tid) {
  constexpr int PER_ROW = HDP / 4;
  constexpr int ROWS_PER_PASS = 256 / PER_ROW;
#pragma unroll
  for (int i = 0; i < HDP / 32; ++i) {
    const int row = tid / PER_ROW + ROWS_PER_PASS * i;
    *reinterpret_cast<floatx4*>(s + row * LD + 4 * (tid % PER_ROW)) = r[i];
  }
}

// Per-lane register operand: row (t0 + lr) of src, d = (HDP/2) hh + s, s < HDP/2.
template <int HDP>
__device__ __forceinline__ void load_reg_operand(float (&f)[HDP / 2], const float* __restrict__ src,
                                                 long long stride, int t, int T, int hd, int hh,
                                                 float scale) {
#pragma unroll
  for (int c = 0; c < HDP / 8; ++c) {
    const int d = (HDP / 2) * hh + 4 * c;
    floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
    if (t < T && d < hd) v = *reinterpret_cast<const floatx4*>(src + (long long)t * stride + d);
    f[4 * c + 0] = v[0] * scale;
    f[4 * c + 1] = v[1] * scale;
    f[4 * c + 2] = v[2] * scale;
    f[4 * c + 3] = v[3] * scale;
  }
}

// acc (+)= X Y^T-style product over d where the LDS tile row (32 rows,
// stride LD) supplies the A operand (row = lr, k = d) and the per-lane
// register array supplies B.  k-slot of step s for lane half hh:
// d = (HDP/2) hh + s.
template <int HDP, int LD>
__device__ __forceinline__ void mma_rows_by_reg(floatx16& acc, const float* __restrict__ s,
                                                const float (&f)[HDP / 2], int lr, int hh) {
#pragma unroll
  for (int c = 0; c < HDP / 8; ++c) {
    const floatx4 a = *reinterpret_cast<const floatx4*>(s + lr * LD + (HDP / 2) * hh + 4 * c);
#pragma unroll
    for (int q = 0; q < 4; ++q) acc = mfma32(a[q], f[4 * c + q], acc);
  }
}

// out^T[d][col] += sum_row X[row][d] * W[row][col] where X is an LDS tile
// [32 rows][LD] and W (32 x 32, rows = k) is held in accumulator layout by the
// lane (column = lr): the MFMA B operand of step s is the lane's register s,
// whose k index is acc_row(s, hh).
template <int HDP, int LD>
__device__ __forceinline__ void mma_tile_T_by_acc(floatx16 (&out)[HDP / 32], const float* __restrict__ s,
                                                  const floatx16& w, int lr, int hh) {
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db)
#pragma unroll
    for (int st = 0; st < 16; ++st) {
      const float a = s[acc_row(st, hh) * LD + 32 * db + lr];
      out[db] = mfma32(a, w[st], out[db]);
    }
}

// Write a wave's 32 x HDP tile held transposed in accumulators (d rows,
// token column lr) to dst rows t0..t0+31 via an LDS staging area [32][HDP+4].
template <int HDP>
__device__ __forceinline__ void store_T_tile(float* __restrict__ stage, const floatx16 (&acc)[HDP / 32],
                                             float scale_by_lane, float* __restrict__ dst,
                                             long long stride, int t0, int T, int hd, int lane) {
  constexpr int LD = HDP + 4;
  const int lr = lane & 31, hh = lane >> 5;
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) stage[lr * LD + 32 * db + acc_row(r, hh)] = acc[db][r] * scale_by_lane;
  __syncthreads();  // called uniformly by the whole block
  constexpr int PER_ROW = HDP / 4;
  for (int e = lane; e < 32 * PER_ROW; e += 64) {
    const int row = e / PER_ROW, d = 4 * (e % PER_ROW);
    const int t = t0 + row;
    if (t < T && d < hd)
      *reinterpret_cast<floatx4*>(dst + (long long)t * stride + d) =
          *reinterpret_cast<const floatx4*>(stage + row * LD + d);
  }
}

// ---------------------------------------------------------------- forward
template <int HDP>
__global__ void __launch_bounds__(256, 2) attn_fwd_kernel(const float* __restrict__ qkv,
                                                          float* __restrict__ out,
                                                          float* __restrict__ lse, AttnShape sh) {
  constexpr int LDK = HDP + 4;   // float4-read tiles
  constexpr int LDV = HDP + 8;   // b32-read tiles (halves 4 rows apart -> other banks)
  constexpr int KSZ = 32 * LDK, VSZ = 32 * LDV;
  __shared__ __attribute__((aligned(16))) float smem[2 * (KSZ + VSZ)];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, hh = lane >> 5;
  const int BH = sh.B * sh.H;
  const int nqt = (sh.T + 127) / 128;
  const int qt = nqt - 1 - (int)(blockIdx.x / BH);  // heaviest tiles first
  const int bh = blockIdx.x % BH;
  const int b = bh / sh.H, h = bh % sh.H;
  const int C = sh.H * sh.hd;
  const long long rs = sh.row_stride;
  const float* qbase = qkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  const float* kbase = qbase + C;
  const float* vbase = qbase + 2 * C;

  const int q0 = qt * 128;
  const int qw0 = q0 + 32 * wave;
  const int my_q = qw0 + lr;
  const float qscale = LOG2E / sqrtf((float)sh.hd);

  float qf[HDP / 2];
  load_reg_operand<HDP>(qf, qbase, rs, my_q, sh.T, sh.hd, hh, qscale);

  floatx16 o[HDP / 32];
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db) zero16(o[db]);
  float m_run = -INFINITY, l_run = 0.f;

  const int last_key = min(sh.T - 1, q0 + 127);
  const int nkb = last_key / 32 + 1;
  const int my_diag = qw0 / 32;  // this wave's diagonal key block

  floatx4 rk[HDP / 32], rv[HDP / 32];
  load_rows<HDP, LDK>(rk, kbase, rs, 0, sh.T, sh.hd, tid);
  load_rows<HDP, LDV>(rv, vbase, rs, 0, sh.T, sh.hd, tid);
  store_rows<HDP, LDK>(smem, rk, tid);
  store_rows<HDP, LDV>(smem + KSZ, rv, tid);
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) {
      load_rows<HDP, LDK>(rk, kbase, rs, (kb + 1) * 32, sh.T, sh.hd, tid);
      load_rows<HDP, LDV>(rv, vbase, rs, (kb + 1) * 32, sh.T, sh.hd, tid);
    }
    if (kb <= my_diag) {
      const float* sK = smem + cur * (KSZ + VSZ);
      const float* sV = sK + KSZ;
      floatx16 s;
      zero16(s);
      mma_rows_by_reg<HDP, LDK>(s, sK, qf, lr, hh);
      const int kv0 = kb * 32;
      const bool need_mask = (kb == my_diag) || (kv0 + 32 > sh.T);
      float bmax = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kv0 + acc_row(r, hh);
        if (need_mask && (key > my_q || key >= sh.T)) s[r] = -INFINITY;
        bmax = fmaxf(bmax, s[r]);
      }
      bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
      const float m_new = fmaxf(m_run, bmax);
      const float alpha = exp2_hw(m_run - m_new);
      float psum = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = exp2_hw(s[r] - m_new);
        psum += s[r];
      }
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < HDP / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      mma_tile_T_by_acc<HDP, LDV>(o, sV, s, lr, hh);
    }
    if (more) {
      float* sN = smem + (cur ^ 1) * (KSZ + VSZ);
      store_rows<HDP, LDK>(sN, rk, tid);
      store_rows<HDP, LDV>(sN + KSZ, rv, tid);
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.f / l_tot;
  if (hh == 0 && my_q < sh.T) lse[(long long)bh * sh.T + my_q] = (m_run + log2f(l_tot)) * LN2;
  float* stage = smem + wave * 32 * (HDP + 4);
  float* obase = out + (long long)b * sh.T * C + (long long)h * sh.hd;
  store_T_tile<HDP>(stage, o, inv, obase, C, qw0, sh.T, sh.hd, lane);
}

// ------------------------------------------------ backward: D and dQ (query-major)
template <int HDP>
__global__ void __launch_bounds__(256, HDP > 64 ? 1 : 2) attn_bwd_dq_kernel(
    const float* __restrict__ dout, const float* __restrict__ qkv, const float* __restrict__ out,
    const float* __restrict__ lse, float* __restrict__ dqkv, float* __restrict__ Dws, AttnShape sh) {
  constexpr int LDK = HDP + 4;  // K: read as float4 (S) and as b32 (dQ)
  constexpr int LDV = HDP + 4;  // V: read as float4 (dP)
  constexpr int KSZ = 32 * LDK, VSZ = 32 * LDV;
  __shared__ __attribute__((aligned(16))) float smem[2 * (KSZ + VSZ)];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, hh = lane >> 5;
  const int BH = sh.B * sh.H;
  const int nqt = (sh.T + 127) / 128;
  const int qt = nqt - 1 - (int)(blockIdx.x / BH);
  const int bh = blockIdx.x % BH;
  const int b = bh / sh.H, h = bh % sh.H;
  const int C = sh.H * sh.hd;
  const long long rs = sh.row_stride;
  const float* qbase = qkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  const float* kbase = qbase + C;
  const float* vbase = qbase + 2 * C;
  const float* dobase = dout + (long long)b * sh.T * C + (long long)h * sh.hd;
  const float* obase = out + (long long)b * sh.T * C + (long long)h * sh.hd;

  const int q0 = qt * 128;
  const int qw0 = q0 + 32 * wave;
  const int my_q = qw0 + lr;
  const float sm_scale = 1.f / sqrtf((float)sh.hd);

  float qf[HDP / 2], dof[HDP / 2];
  load_reg_operand<HDP>(qf, qbase, rs, my_q, sh.T, sh.hd, hh, LOG2E * sm_scale);
  load_reg_operand<HDP>(dof, dobase, C, my_q, sh.T, sh.hd, hh, 1.f);
  float Dq;
  {
    float of[HDP / 2];
    load_reg_operand<HDP>(of, obase, C, my_q, sh.T, sh.hd, hh, 1.f);
    float part = 0.f;
#pragma unroll
    for (int s = 0; s < HDP / 2; ++s) part += dof[s] * of[s];
    Dq = part + __shfl_xor(part, 32, 64);
  }
  if (hh == 0 && my_q < sh.T) Dws[(long long)bh * sh.T + my_q] = Dq;
  const float lse2 = my_q < sh.T ? lse[(long long)bh * sh.T + my_q] * LOG2E : 0.f;

  floatx16 dq[HDP / 32];
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db) zero16(dq[db]);

  const int last_key = min(sh.T - 1, q0 + 127);
  const int nkb = last_key / 32 + 1;
  const int my_diag = qw0 / 32;

  floatx4 rk[HDP / 32], rv[HDP / 32];
  load_rows<HDP, LDK>(rk, kbase, rs, 0, sh.T, sh.hd, tid);
  load_rows<HDP, LDV>(rv, vbase, rs, 0, sh.T, sh.hd, tid);
  store_rows<HDP, LDK>(smem, rk, tid);
  store_rows<HDP, LDV>(smem + KSZ, rv, tid);
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) {
      load_rows<HDP, LDK>(rk, kbase, rs, (kb + 1) * 32, sh.T, sh.hd, tid);
      load_rows<HDP, LDV>(rv, vbase, rs, (kb + 1) * 32, sh.T, sh.hd, tid);
    }
    if (kb <= my_diag) {
      const float* sK = smem + cur * (KSZ + VSZ);
      const float* sV = sK + KSZ;
      floatx16 s, dp;
      zero16(s);
      zero16(dp);
      mma_rows_by_reg<HDP, LDK>(s, sK, qf, lr, hh);    // S^T  [key][q]
      mma_rows_by_reg<HDP, LDV>(dp, sV, dof, lr, hh);  // dP^T [key][q]
      const int kv0 = kb * 32;
      const bool need_mask = (kb == my_diag) || (kv0 + 32 > sh.T);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kv0 + acc_row(r, hh);
        float p = exp2_hw(s[r] - lse2);
        if (need_mask && (key > my_q || key >= sh.T)) p = 0.f;
        s[r] = p * (dp[r] - Dq);  // dS^T
      }
      mma_tile_T_by_acc<HDP, LDK>(dq, sK, s, lr, hh);  // dQ^T[d][q] += K^T dS^T
    }
    if (more) {
      float* sN = smem + (cur ^ 1) * (KSZ + VSZ);
      store_rows<HDP, LDK>(sN, rk, tid);
      store_rows<HDP, LDV>(sN + KSZ, rv, tid);
    }
    __syncthreads();
  }
  float* stage = smem + wave * 32 * (HDP + 4);
  float* dqbase = dqkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  store_T_tile<HDP>(stage, dq, sm_scale, dqbase, rs, qw0, sh.T, sh.hd, lane);
}

// ------------------------------------------------ backward: D = rowsum(dO o O)
// One block per token row (b, t) at a time: the block reads the row's H hd
// floats of dO and O once, coalesced, stores the float4 partial dots in LDS
// (C / 4 floats of dynamic shared memory) and thread h adds up head h's
// hd / 4 partials in order.  D laid out [B, H, T].
__global__ void __launch_bounds__(256) attn_bwd_d_kernel(const float* __restrict__ dout,
                                                         const float* __restrict__ out,
                                                         float* __restrict__ D, int B, int T, int H,
                                                         int hd) {
  extern __shared__ float part[];
  const int C4 = H * hd / 4, hq = hd / 4;
  const long long rows = (long long)B * T;
  for (long long row = blockIdx.x; row < rows; row += gridDim.x) {
    const floatx4* g = reinterpret_cast<const floatx4*>(dout + row * H * hd);
    const floatx4* o = reinterpret_cast<const floatx4*>(out + row * H * hd);
    for (int i = threadIdx.x; i < C4; i += 256) {
      const floatx4 a = g[i], c = o[i];
      part[i] = (a[0] * c[0] + a[1] * c[1]) + (a[2] * c[2] + a[3] * c[3]);
    }
    __syncthreads();
    const int b = (int)(row / T), t = (int)(row % T);
    for (int h = threadIdx.x; h < H; h += 256) {
      float acc = 0.f;
      for (int j = 0; j < hq; ++j) acc += part[h * hq + j];
      D[((long long)b * H + h) * T + t] = acc;
    }
    __syncthreads();
  }
}

// ------------------------------------------------ backward: dK and dV (key-major)
template <int HDP>
__global__ void __launch_bounds__(256, 1) attn_bwd_dkv_kernel(
    const float* __restrict__ dout, const float* __restrict__ qkv, const float* __restrict__ lse,
    const float* __restrict__ Dws, float* __restrict__ dqkv, float* __restrict__ dS, AttnShape sh) {
  constexpr int LD = HDP + 4;
  constexpr int TSZ = 32 * LD;
  // per buffer: Q tile, dO tile, lse2[32], D[32]
  constexpr int BUF = 2 * TSZ + 64;
  __shared__ __attribute__((aligned(16))) float smem[2 * BUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, hh = lane >> 5;
  const int BH = sh.B * sh.H;
  const int kt = (int)(blockIdx.x / BH);  // low key tiles see the most queries: first
  const int bh = blockIdx.x % BH;
  const int b = bh / sh.H, h = bh % sh.H;
  const int C = sh.H * sh.hd;
  const long long rs = sh.row_stride;
  const float* qbase = qkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  const float* kbase = qbase + C;
  const float* vbase = qbase + 2 * C;
  const float* dobase = dout + (long long)b * sh.T * C + (long long)h * sh.hd;
  const float* lrow = lse + (long long)bh * sh.T;
  const float* drow = Dws + (long long)bh * sh.T;

  const int k0 = kt * 128;
  const int kw0 = k0 + 32 * wave;
  const int my_k = kw0 + lr;
  const float sm_scale = 1.f / sqrtf((float)sh.hd);
  // dS / sqrt(hd) for the dQ product, [B, H, T, T], column my_k of this lane
  float* ds_col = dS ? dS + (long long)bh * sh.T * sh.T + my_k : nullptr;
  const bool ds_lane = my_k < sh.T;

  float kf[HDP / 2], vf[HDP / 2];
  load_reg_operand<HDP>(kf, kbase, rs, my_k, sh.T, sh.hd, hh, LOG2E * sm_scale);
  load_reg_operand<HDP>(vf, vbase, rs, my_k, sh.T, sh.hd, hh, 1.f);

  floatx16 dk[HDP / 32], dv[HDP / 32];
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db) {
    zero16(dk[db]);
    zero16(dv[db]);
  }

  const int qb0 = k0 / 32;                // first query block touching this key tile
  const int nqb = (sh.T + 31) / 32;
  const int my_first = kw0 / 32;          // this wave's diagonal query block

  floatx4 rq[HDP / 32], rdo[HDP / 32];
  float rl = 0.f, rd = 0.f;
  auto load_q = [&](int qb) {
    load_rows<HDP, LD>(rq, qbase, rs, qb * 32, sh.T, sh.hd, tid);
    load_rows<HDP, LD>(rdo, dobase, C, qb * 32, sh.T, sh.hd, tid);
    if (tid < 32) {
      const int t = qb * 32 + tid;
      rl = t < sh.T ? lrow[t] * LOG2E : INFINITY;  // rows past T give P = 0
      rd = t < sh.T ? drow[t] : 0.f;
    }
  };
  auto store_q = [&](float* sb) {
    store_rows<HDP, LD>(sb, rq, tid);
    store_rows<HDP, LD>(sb + TSZ, rdo, tid);
    if (tid < 32) {
      sb[2 * TSZ + tid] = rl;
      sb[2 * TSZ + 32 + tid] = rd;
    }
  };
  if (qb0 < nqb) {
    load_q(qb0);
    store_q(smem);
  }
  __syncthreads();

  for (int qb = qb0; qb < nqb; ++qb) {
    const int cur = (qb - qb0) & 1;
    const bool more = qb + 1 < nqb;
    if (more) load_q(qb + 1);
    if (qb >= my_first && kw0 < sh.T) {
      const float* sQ = smem + cur * BUF;
      const float* sdO = sQ + TSZ;
      const float* sl = sQ + 2 * TSZ;
      const float* sd = sl + 32;
      floatx16 s, dp;
      zero16(s);
      zero16(dp);
      mma_rows_by_reg<HDP, LD>(s, sQ, kf, lr, hh);    // S  [q][key]
      mma_rows_by_reg<HDP, LD>(dp, sdO, vf, lr, hh);  // dP [q][key]
      const int qv0 = qb * 32;
      const bool need_mask = (qb == my_first) || (my_k >= sh.T);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qi = acc_row(r, hh);
        float p = exp2_hw(s[r] - sl[qi]);
        if (need_mask && (my_k > qv0 + qi || my_k >= sh.T)) p = 0.f;
        s[r] = p;
        dp[r] = p * (dp[r] - sd[qi]);
      }
      mma_tile_T_by_acc<HDP, LD>(dv, sdO, s, lr, hh);  // dV^T[d][key] += dO^T P
      mma_tile_T_by_acc<HDP, LD>(dk, sQ, dp, lr, hh);  // dK^T[d][key] += Q^T dS
      if (ds_col && ds_lane) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int q = qv0 + acc_row(r, hh);
          if (q < sh.T) ds_col[(long long)q * sh.T] = dp[r] * sm_scale;
        }
      }
    } else if (ds_col && ds_lane && qb < my_first) {
      // query blocks of the diagonal 128-row tile that precede this wave's
      // keys: fully masked, stored as zeros because the dQ product of that
      // tile sums keys up to the tile's end
      const int qv0 = qb * 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int q = qv0 + acc_row(r, hh);
        if (q < sh.T) ds_col[(long long)q * sh.T] = 0.f;
      }
    }
    if (more) store_q(smem + (cur ^ 1) * BUF);
    __syncthreads();
  }
  float* stage = smem + wave * 32 * (HDP + 4);
  float* dkbase = dqkv + (long long)b * sh.T * rs + (long long)h * sh.hd + C;
  store_T_tile<HDP>(stage, dk, sm_scale, dkbase, rs, kw0, sh.T, sh.hd, lane);
  __syncthreads();
  store_T_tile<HDP>(stage, dv, 1.f, dkbase + C, rs, kw0, sh.T, sh.hd, lane);
}

bt_status check_attn(const void* a, const void* b2, int B, int T, int H, int hd, const char* who) {
  BT_RETURN_IF(B < 1 || T < 1 || H < 1, BT_ESHAPE, "%s: B=%d T=%d H=%d must be >= 1", who, B, T, H);
  BT_RETURN_IF(hd < 4 || hd > 128 || (hd & 3), BT_ESHAPE,
               "%s: head dim %d unsupported (multiple of 4, <= 128)", who, hd);
  BT_RETURN_IF(!a || !b2, BT_EINVAL, "%s: NULL pointer", who);
  BT_RETURN_IF((long long)B * H * ((T + 127) / 128) > 0x7fffffffLL, BT_ESHAPE, "%s: grid too large", who);
  return BT_OK;
}

}  // namespace
}  // namespace bt

using namespace bt;

extern "C" bt_status bt_attention_fwd(const float* qkv, float* out, float* lse, int B, int T, int H,
                                      int hd, void* stream) {
  BT_TRY(check_attn(qkv, out, B, T, H, hd, "bt_attention_fwd"));
  BT_RETURN_IF(!lse, BT_EINVAL, "bt_attention_fwd: lse is NULL");
  BT_RETURN_IF(!aligned16(qkv) || !aligned16(out), BT_EALIGN, "bt_attention_fwd: qkv/out must be 16-byte aligned");
  AttnShape sh{B, T, H, hd, 3LL * H * hd};
  dim3 grid((unsigned)(B * H * ((T + 127) / 128)));
  hipStream_t s = as_stream(stream);
  if (hd <= 32)
    hipLaunchKernelGGL(attn_fwd_kernel<32>, grid, dim3(256), 0, s, qkv, out, lse, sh);
  else if (hd <= 64)
    hipLaunchKernelGGL(attn_fwd_kernel<64>, grid, dim3(256), 0, s, qkv, out, lse, sh);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<128>, grid, dim3(256), 0, s, qkv, out, lse, sh);
  return check_launch("attn_fwd_kernel");
}

extern "C" size_t bt_attention_bwd_ws_min_bytes(int B, int T, int H, int hd) {
  (void)hd;
  if (B <= 0 || T <= 0 || H <= 0) return 0;
  return align_up((size_t)B * H * T * sizeof(float), 256);
}

// The stored-dS backward reads dS rows as float4 along the keys: T % 4 == 0.
bool attn_stores_ds(int T) { return T % 4 == 0; }

extern "C" size_t bt_attention_bwd_ws_bytes(int B, int T, int H, int hd) {
  if (B <= 0 || T <= 0 || H <= 0) return 0;
  const size_t base = bt_attention_bwd_ws_min_bytes(B, T, H, hd);
  if (!attn_stores_ds(T)) return base;
  return base + align_up((size_t)B * H * T * T * sizeof(float), 256);
}

extern "C" bt_status bt_attention_bwd(const float* dout, const float* qkv, const float* out,
                                      const float* lse, float* dqkv, void* ws, size_t ws_bytes, int B,
                                      int T, int H, int hd, void* stream) {
  BT_TRY(check_attn(qkv, dout, B, T, H, hd, "bt_attention_bwd"));
  BT_RETURN_IF(!out || !lse || !dqkv, BT_EINVAL, "bt_attention_bwd: NULL pointer");
  BT_RETURN_IF(!aligned16(qkv) || !aligned16(out) || !aligned16(dout) || !aligned16(dqkv), BT_EALIGN,
               "bt_attention_bwd: tensors must be 16-byte aligned");
  BT_RETURN_IF(dqkv == qkv, BT_EINVAL, "bt_attention_bwd: dqkv must not alias qkv");
  const size_t need_min = bt_attention_bwd_ws_min_bytes(B, T, H, hd);
  BT_RETURN_IF(!ws || ws_bytes < need_min, BT_EWORKSPACE,
               "bt_attention_bwd: workspace of %zu bytes needed (got %zu)", need_min, ws_bytes);
  BT_RETURN_IF(!aligned16(ws), BT_EALIGN, "bt_attention_bwd: workspace must be 16-byte aligned");
  AttnShape sh{B, T, H, hd, 3LL * H * hd};
  float* D = static_cast<float*>(ws);
  dim3 gq((unsigned)(B * H * ((T + 127) / 128)));
  hipStream_t s = as_stream(stream);
  if (attn_stores_ds(T) && ws_bytes >= bt_attention_bwd_ws_bytes(B, T, H, hd)) {
    // D, then dK/dV with dS stored, then dQ = dS K (scale folded into dS)
    float* dS = reinterpret_cast<float*>(static_cast<char*>(ws) + need_min);
    const long long rows = (long long)B * T;
    const unsigned gd = (unsigned)(rows < 8192 ? rows : 8192);
    const size_t part_bytes = (size_t)H * hd / 4 * sizeof(float);
    BT_RETURN_IF(part_bytes > 64 * 1024, BT_ESHAPE, "bt_attention_bwd: H * hd = %d too large", H * hd);
    hipLaunchKernelGGL(attn_bwd_d_kernel, dim3(gd), dim3(256), part_bytes, s, dout, out, D, B, T, H, hd);
    BT_TRY(check_launch("attn_bwd_d_kernel"));
    if (hd <= 32)
      hipLaunchKernelGGL(attn_bwd_dkv_kernel<32>, gq, dim3(256), 0, s, dout, qkv, lse, D, dqkv, dS, sh);
    else if (hd <= 64)
      hipLaunchKernelGGL(attn_bwd_dkv_kernel<64>, gq, dim3(256), 0, s, dout, qkv, lse, D, dqkv, dS, sh);
    else
      hipLaunchKernelGGL(attn_bwd_dkv_kernel<128>, gq, dim3(256), 0, s, dout, qkv, lse, D, dqkv, dS, sh);
    BT_TRY(check_launch("attn_bwd_dkv_kernel"));
    const long long rs = sh.row_stride;
    // per (b, h): dQ [T][hd] (rows of dqkv, stride 3 H hd) = dS [T][T] K [T][hd]
    return gemm_causal_batched(T, hd, T, dS, T, (long long)H * T * T, (long long)T * T,
                               qkv + (long long)H * hd, (int)rs, (long long)T * rs, hd,
                               dqkv, (int)rs, (long long)T * rs, hd, B, H, s);
  }
  if (hd <= 32) {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<32>, gq, dim3(256), 0, s, dout, qkv, out, lse, dqkv, D, sh);
    BT_TRY(check_launch("attn_bwd_dq_kernel"));
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<32>, gq, dim3(256), 0, s, dout, qkv, lse, D, dqkv, nullptr, sh);
  } else if (hd <= 64) {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<64>, gq, dim3(256), 0, s, dout, qkv, out, lse, dqkv, D, sh);
    BT_TRY(check_launch("attn_bwd_dq_kernel"));
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<64>, gq, dim3(256), 0, s, dout, qkv, lse, D, dqkv, nullptr, sh);
  } else {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<128>, gq, dim3(256), 0, s, dout, qkv, out, lse, dqkv, D, sh);
    BT_TRY(check_launch("attn_bwd_dq_kernel"));
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<128>, gq, dim3(256), 0, s, dout, qkv, lse, D, dqkv, nullptr, sh);
  }
  return check_launch("attn_bwd_dkv_kernel");
}
