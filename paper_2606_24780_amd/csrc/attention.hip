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
//    LDS and shared by the 4 waves.  The forward at head dim 64 with full key
//    tiles copies its key and value tiles straight into swizzled LDS tiles
//    (global_load_lds_dwordx4, scalar tile base); elsewhere tiles are staged
//    through registers into padded LDS tiles.
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
//
// Context parallelism (section "Context Parallelism"): the same kernels, in
// their SEG instantiation, compute one rank's share of ring attention.  The
// local query rows and the key/value rows of the shard the rank holds are each
// one or two contiguous segments of global token positions, and visibility
// is decided by position (key visible iff its position <= the query's).
// Every 32-row wave tile and 32-row streamed tile then covers consecutive
// positions, so a tile pair is either fully visible, fully masked (skipped)
// or on the diagonal (masked per element), as in the plain causal case.  The
// forward can fold its result into the running (out, lse) with the
// sigmoid-form update in its epilogue; the backward takes the final lse and
// D and adds its dQ and the shard's dK/dV into accumulators.
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

// One rank's share under context parallelism (SEG kernels only).  Rows of the
// query side (T of AttnShape) and of the key/value side (Tk) are 1 or 2
// segments of `seg` rows; segment i starts at global position q_pos[i] /
// k_pos[i] (multiples of 32; seg a multiple of 128).
struct AttnSegs {
  const float* kv;      // K row t at kv + t kv_stride, V at + H hd
  float* dkv;           // gradient of the shard, same layout
  long long kv_stride;  // token stride of kv and dkv
  int Tk, seg;
  int q_pos[2], k_pos[2];
  int flags;            // forward: merge; backward: ACC_DQ | ACC_DKV
};
constexpr int SEG_MERGE = 1, SEG_ACC_DQ = 1, SEG_ACC_DKV = 2;

// Global position of row `row` of a segmented side.
__device__ __forceinline__ int seg_pos(const int (&pos)[2], int seg, int row) {
  return row < seg ? pos[0] + row : pos[1] + (row - seg);
}

// Streamed 32-row tiles needed by a tile of queries whose last position is
// `qlast`: in each key segment the visible tiles are a prefix.
__device__ __forceinline__ int seg_prefix_tiles(int qlast, int kpos0, int seg) {
  if (qlast < kpos0) return 0;
  return min(seg / 32, (qlast - kpos0) / 32 + 1);
}

// Streamed 32-row query tiles needed by a tile of keys whose first position is
// `kfirst`: in each query segment they are a suffix; returns its first tile.
__device__ __forceinline__ int seg_suffix_first(int kfirst, int qpos0) {
  const int a = kfirst - 31 - qpos0;
  return a > 0 ? (a + 31) / 32 : 0;
}

// Rows [r0, r0 + 32) of one of the Q/K/V/dO-like matrices (src points at
// (b, token 0, head h), `stride` is the token stride) into registers, HDP/4
// float4 per row over 256 threads, without branches: rows past T and columns
// past hd read the last valid row / column group instead (always in bounds,
// T >= 1, hd >= 4), and store_rows_masked zeroes them when the tile goes to
// an LDS tile [32][LD].  No register is written between issuing the loads
// and their use, so the only wait for them is the one before the LDS store.
template <int HDP>
__device__ __forceinline__ void load_rows_clamped(floatx4 (&r)[HDP / 32], const float* __restrict__ src,
                                                  long long stride, int r0, int T, int hd, int tid) {
  constexpr int PER_ROW = HDP / 4;
  constexpr int ROWS_PER_PASS = 256 / PER_ROW;
#pragma unroll
  for (int i = 0; i < HDP / 32; ++i) {
    const int t = min(r0 + tid / PER_ROW + ROWS_PER_PASS * i, T - 1);
    const int d = min(4 * (tid % PER_ROW), hd - 4);
    r[i] = *reinterpret_cast<const floatx4*>(src + (long long)t * stride + d);
  }
}

template <int HDP, int LD>
__device__ __forceinline__ void store_rows_masked(float* __restrict__ s, const floatx4 (&r)[HDP / 32], int tid,
                                                  int r0, int T, int hd) {
  constexpr int PER_ROW = HDP / 4;
  constexpr int ROWS_PER_PASS = 256 / PER_ROW;
#pragma unroll
  for (int i = 0; i < HDP / 32; ++i) {
    const int row = tid / PER_ROW + ROWS_PER_PASS * i;
    const int d = 4 * (tid % PER_ROW);
    const bool ok = r0 + row < T && d < hd;
    *reinterpret_cast<floatx4*>(s + row * LD + d) = ok ? r[i] : floatx4{0.f, 0.f, 0.f, 0.f};
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
__device__ __forceinline__ void stage_T_tile(float* __restrict__ stage, const floatx16 (&acc)[HDP / 32],
                                             float scale_by_lane, int lane) {
  constexpr int LD = HDP + 4;
  const int lr = lane & 31, hh = lane >> 5;
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) stage[lr * LD + 32 * db + acc_row(r, hh)] = acc[db][r] * scale_by_lane;
}

// `add`: dst += tile instead of dst = tile (uniform across the block).
template <int HDP>
__device__ __forceinline__ void store_T_tile(float* __restrict__ stage, const floatx16 (&acc)[HDP / 32],
                                             float scale_by_lane, float* __restrict__ dst,
                                             long long stride, int t0, int T, int hd, int lane,
                                             bool add = false) {
  constexpr int LD = HDP + 4;
  stage_T_tile<HDP>(stage, acc, scale_by_lane, lane);
  __syncthreads();  // called uniformly by the whole block
  constexpr int PER_ROW = HDP / 4;
  for (int e = lane; e < 32 * PER_ROW; e += 64) {
    const int row = e / PER_ROW, d = 4 * (e % PER_ROW);
    const int t = t0 + row;
    if (t < T && d < hd) {
      floatx4* g = reinterpret_cast<floatx4*>(dst + (long long)t * stride + d);
      floatx4 v = *reinterpret_cast<const floatx4*>(stage + row * LD + d);
      if (add) v += *g;
      *g = v;
    }
  }
}

// The running state's update by one partial result, for one row (section
// "Context Parallelism": out <- out - sigmoid(blse - lse) (out - bout),
// lse <- lse - log sigmoid(lse - blse)).  Returns the weight of the block in
// the new output, or the markers KEEP (block empty: state unchanged) and TAKE
// (state empty: the block replaces it); *new_lse receives the merged lse.
constexpr float MERGE_KEEP = -1.f, MERGE_TAKE = 2.f;
__device__ __forceinline__ float lse_merge_row(float lse, float blse, float* new_lse) {
  if (blse == -INFINITY) {
    *new_lse = lse;
    return MERGE_KEEP;
  }
  if (lse == -INFINITY) {
    *new_lse = blse;
    return MERGE_TAKE;
  }
  const float x = blse - lse;
  const float z = expf(-fabsf(x));
  const float sig = x >= 0.f ? 1.f / (1.f + z) : z / (1.f + z);  // sigmoid(blse - lse)
  // -log sigmoid(lse - blse) = softplus(blse - lse) = max(x, 0) + log1p(e^-|x|)
  *new_lse = lse + (fmaxf(x, 0.f) + log1pf(z));
  return sig;
}

__device__ __forceinline__ floatx4 lse_merge_apply(float w, const floatx4& o, const floatx4& b) {
  if (w == MERGE_TAKE) return b;
  return o - w * (o - b);
}

// Forward epilogue that folds the wave's 32 x HDP result (normalised by
// scale_by_lane) into the running out/lse rows t0..t0+31.  wts: 32 floats of
// LDS for the wave.
template <int HDP>
__device__ __forceinline__ void store_T_tile_merge(float* __restrict__ stage, float* __restrict__ wts,
                                                   const floatx16 (&acc)[HDP / 32], float scale_by_lane,
                                                   float blse, float* __restrict__ dst, long long stride,
                                                   float* __restrict__ lse_row, int t0, int T, int hd,
                                                   int lane) {
  constexpr int LD = HDP + 4;
  const int lr = lane & 31, hh = lane >> 5;
  stage_T_tile<HDP>(stage, acc, scale_by_lane, lane);
  if (hh == 0) {
    float w = MERGE_KEEP;
    if (t0 + lr < T) {
      float nl;
      w = lse_merge_row(lse_row[t0 + lr], blse, &nl);
      lse_row[t0 + lr] = nl;
    }
    wts[lr] = w;
  }
  __syncthreads();  // called uniformly by the whole block
  constexpr int PER_ROW = HDP / 4;
  for (int e = lane; e < 32 * PER_ROW; e += 64) {
    const int row = e / PER_ROW, d = 4 * (e % PER_ROW);
    const int t = t0 + row;
    const float w = wts[row];
    if (t < T && d < hd && w != MERGE_KEEP) {
      floatx4* g = reinterpret_cast<floatx4*>(dst + (long long)t * stride + d);
      const floatx4 b = *reinterpret_cast<const floatx4*>(stage + row * LD + d);
      *g = lse_merge_apply(w, w == MERGE_TAKE ? b : *g, b);
    }
  }
}

// ---------------------------------------------------- direct-to-LDS tiles
// The forward's key and value tiles at head dim 64 when every key tile is
// full: unpadded [32][64] tiles copied straight from global memory into LDS
// (global_load_lds_dwordx4: a wave instruction moves 1 KB = 4 rows, lane i
// landing at byte 16 i; a tile is 8 such slices, 2 per wave).  No staging
// registers, no LDS stores, and every address is a scalar tile base plus a
// per-lane offset fixed for the whole kernel.  The source of each lane is
// chosen so the tiles are stored swizzled instead of padded:
//  * keys (read as float4 along d by 32 consecutive rows): the 16-byte chunk
//    c of row r is stored at chunk c ^ (r & 15), so the 16 rows a quarter
//    wave reads land on 16 different bank groups;
//  * values (read as b32 by 32 consecutive columns, the two lane halves 4
//    rows apart): rows with bit 2 set have their two 32-column halves
//    swapped, so the two halves of a wave read different banks.
__device__ __forceinline__ void fwd_copy_offsets(unsigned (&ok)[2], unsigned (&ov)[2], long long ks, int wave,
                                                 int lane) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 4 * (2 * wave + j) + lane / 16;
    const int c4 = 4 * (lane % 16);  // LDS column of this lane's 16 bytes
    ok[j] = (unsigned)((row * ks + 4 * ((c4 / 4) ^ (row & 15))) * 4);
    ov[j] = (unsigned)((row * ks + (c4 ^ (((row >> 2) & 1) << 5))) * 4);
  }
}

// S = (rows of the swizzled key tile) x (register operand), as
// mma_rows_by_reg<64, ...> on an unpadded tile.
__device__ __forceinline__ void mma_rows_by_reg_swz(floatx16& acc, const float* __restrict__ s,
                                                    const float (&f)[32], int lr, int hh) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const floatx4 a = *reinterpret_cast<const floatx4*>(s + lr * 64 + 4 * ((8 * hh + c) ^ (lr & 15)));
#pragma unroll
    for (int q = 0; q < 4; ++q) acc = mfma32(a[q], f[4 * c + q], acc);
  }
}

// out^T += (swizzled value tile)^T x w, as mma_tile_T_by_acc<64, ...>:
// register st of lane half hh holds row acc_row(st, hh), whose bit 2 is hh.
__device__ __forceinline__ void mma_tile_T_by_acc_swz(floatx16 (&out)[2], const float* __restrict__ s,
                                                      const floatx16& w, int lr, int hh) {
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int st = 0; st < 16; ++st) {
      const float a = s[acc_row(st, hh) * 64 + ((32 * db + lr) ^ (hh << 5))];
      out[db] = mfma32(a, w[st], out[db]);
    }
}

// ---------------------------------------------------------------- forward
// SEG: one rank's share (keys from sg.kv, visibility by segment positions,
// optional merge into the running out/lse).
template <int HDP, bool SEG, bool DTL = false>
__global__ void __launch_bounds__(256, 2) attn_fwd_kernel(const float* __restrict__ qkv,
                                                          float* __restrict__ out,
                                                          float* __restrict__ lse, AttnShape sh,
                                                          AttnSegs sg) {
  constexpr int LDK = HDP + 4;   // float4-read tiles
  constexpr int LDV = HDP + 8;   // b32-read tiles (halves 4 rows apart -> other banks)
  constexpr int KSZ = 32 * LDK, VSZ = 32 * LDV;
  __shared__ __attribute__((aligned(16))) float smem[2 * (KSZ + VSZ)];
  static_assert(4 * 32 * (HDP + 4) + 4 * 32 <= 2 * (KSZ + VSZ), "epilogue staging must fit");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, hh = lane >> 5;
  const int BH = sh.B * sh.H;
  const int nqt = (sh.T + 127) / 128;
  const int qt = nqt - 1 - (int)(blockIdx.x / BH);  // heaviest tiles first
  const int bh = blockIdx.x % BH;
  const int b = bh / sh.H, h = bh % sh.H;
  const int C = sh.H * sh.hd;
  const long long rs = sh.row_stride;
  const int Tk = SEG ? sg.Tk : sh.T;
  const long long ks = SEG ? sg.kv_stride : rs;
  const float* qbase = qkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  const float* kbase = SEG ? sg.kv + (long long)b * Tk * ks + (long long)h * sh.hd : qbase + C;
  const float* vbase = kbase + C;

  const int q0 = qt * 128;
  const int qw0 = q0 + 32 * wave;
  const int my_q = qw0 + lr;
  // positions: the block's 128 rows lie in one segment
  const int qp0 = SEG ? seg_pos(sg.q_pos, sg.seg, q0) : q0;
  const int wpos = qp0 + 32 * wave;  // this wave's first query position
  const int my_qpos = wpos + lr;
  const float qscale = LOG2E / sqrtf((float)sh.hd);

  float qf[HDP / 2];
  load_reg_operand<HDP>(qf, qbase, rs, my_q, sh.T, sh.hd, hh, qscale);

  floatx16 o[HDP / 32];
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db) zero16(o[db]);
  float m_run = -INFINITY, l_run = 0.f;

  // streamed key tiles: causal, a prefix of the rows; SEG, a prefix of each
  // key segment (n0 tiles of the first)
  int nkb, n0;
  if (SEG) {
    n0 = seg_prefix_tiles(qp0 + 127, sg.k_pos[0], sg.seg);
    nkb = n0 + (Tk > sg.seg ? seg_prefix_tiles(qp0 + 127, sg.k_pos[1], sg.seg) : 0);
  } else {
    nkb = min(sh.T - 1, q0 + 127) / 32 + 1;
    n0 = nkb;
  }
  auto key_row = [&](int kb) { return SEG ? (kb < n0 ? 32 * kb : sg.seg + 32 * (kb - n0)) : 32 * kb; };
  auto key_pos = [&](int kb) { return SEG ? (kb < n0 ? sg.k_pos[0] + 32 * kb : sg.k_pos[1] + 32 * (kb - n0)) : 32 * kb; };

  floatx4 rk[HDP / 32], rv[HDP / 32];
  // DTL: key and value tiles copied straight into LDS (below)
  unsigned ok_[2], ov_[2];
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) float*)smem;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  if constexpr (DTL) fwd_copy_offsets(ok_, ov_, ks, wave_u, lane);
  auto issue = [&](int kb, int buf) {
    const long long r0 = key_row(kb);
    const unsigned l = lds0 + 4u * buf * (KSZ + VSZ) + 2048u * wave_u;
#pragma unroll
    for (int j = 0; j < 2; ++j) copy16_to_lds_sbase(kbase + r0 * ks, ok_[j], l + 1024u * j);
#pragma unroll
    for (int j = 0; j < 2; ++j) copy16_to_lds_sbase(vbase + r0 * ks, ov_[j], l + 4u * KSZ + 1024u * j);
  };
  if (nkb > 0) {
    if constexpr (DTL) {
      issue(0, 0);
      wait_copies();
    } else {
      load_rows_clamped<HDP>(rk, kbase, ks, key_row(0), Tk, sh.hd, tid);
      load_rows_clamped<HDP>(rv, vbase, ks, key_row(0), Tk, sh.hd, tid);
      store_rows_masked<HDP, LDK>(smem, rk, tid, key_row(0), Tk, sh.hd);
      store_rows_masked<HDP, LDV>(smem + KSZ, rv, tid, key_row(0), Tk, sh.hd);
    }
  }
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) {
      if constexpr (DTL) {
        issue(kb + 1, cur ^ 1);  // the other buffer was last read before the previous barrier
      } else {
        load_rows_clamped<HDP>(rk, kbase, ks, key_row(kb + 1), Tk, sh.hd, tid);
        load_rows_clamped<HDP>(rv, vbase, ks, key_row(kb + 1), Tk, sh.hd, tid);
      }
    }
    const int kp0 = key_pos(kb);
    if (kp0 <= wpos + 31) {  // some key of the tile visible to this wave
      const float* sK = smem + cur * (KSZ + VSZ);
      const float* sV = sK + KSZ;
      floatx16 s;
      zero16(s);
      if constexpr (DTL)
        mma_rows_by_reg_swz(s, sK, qf, lr, hh);
      else
        mma_rows_by_reg<HDP, LDK>(s, sK, qf, lr, hh);
      const int kr0 = key_row(kb);
      if ((kp0 + 31 > wpos) || (kr0 + 32 > Tk)) {  // diagonal or ragged tile (uniform)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kk = acc_row(r, hh);
          const bool dead = (kp0 + kk > my_qpos) | (kr0 + kk >= Tk);
          s[r] = dead ? -INFINITY : s[r];
        }
      }
      float bmax = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) bmax = fmaxf(bmax, s[r]);
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
      if constexpr (DTL)
        mma_tile_T_by_acc_swz(o, sV, s, lr, hh);
      else
        mma_tile_T_by_acc<HDP, LDV>(o, sV, s, lr, hh);
    }
    if constexpr (DTL) {
      wait_copies();
    } else if (more) {
      float* sN = smem + (cur ^ 1) * (KSZ + VSZ);
      store_rows_masked<HDP, LDK>(sN, rk, tid, key_row(kb + 1), Tk, sh.hd);
      store_rows_masked<HDP, LDV>(sN + KSZ, rv, tid, key_row(kb + 1), Tk, sh.hd);
    }
    __syncthreads();
  }

  // A query that saw no key (possible only across shards) keeps l = 0:
  // output 0, lse -inf.
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const bool seen = l_tot > 0.f;
  const float inv = seen ? 1.f / l_tot : 0.f;
  const float row_lse = seen ? (m_run + log2f(l_tot)) * LN2 : -INFINITY;
  float* stage = smem + wave * 32 * (HDP + 4);
  float* obase = out + (long long)b * sh.T * C + (long long)h * sh.hd;
  if (SEG && (sg.flags & SEG_MERGE)) {
    float* wts = smem + 4 * 32 * (HDP + 4) + 32 * wave;
    store_T_tile_merge<HDP>(stage, wts, o, inv, row_lse, obase, C, lse + (long long)bh * sh.T, qw0, sh.T,
                            sh.hd, lane);
  } else {
    if (hh == 0 && my_q < sh.T) lse[(long long)bh * sh.T + my_q] = row_lse;
    store_T_tile<HDP>(stage, o, inv, obase, C, qw0, sh.T, sh.hd, lane);
  }
}

// ------------------------------------------------ backward: D and dQ (query-major)
// Causal: computes D = rowsum(dO o O) for its rows and stores it to Dws for
// the key-major kernel.  SEG: reads D from Dws (the final output's row sums,
// computed once per rank), keys from sg.kv, optional dQ accumulation.
template <int HDP, bool SEG>
__global__ void __launch_bounds__(256, HDP > 64 ? 1 : 2) attn_bwd_dq_kernel(
    const float* __restrict__ dout, const float* __restrict__ qkv, const float* __restrict__ out,
    const float* __restrict__ lse, float* __restrict__ dqkv, float* __restrict__ Dws, AttnShape sh,
    AttnSegs sg) {
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
  const int Tk = SEG ? sg.Tk : sh.T;
  const long long ks = SEG ? sg.kv_stride : rs;
  const float* qbase = qkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  const float* kbase = SEG ? sg.kv + (long long)b * Tk * ks + (long long)h * sh.hd : qbase + C;
  const float* vbase = kbase + C;
  const float* dobase = dout + (long long)b * sh.T * C + (long long)h * sh.hd;

  const int q0 = qt * 128;
  const int qw0 = q0 + 32 * wave;
  const int my_q = qw0 + lr;
  const int qp0 = SEG ? seg_pos(sg.q_pos, sg.seg, q0) : q0;
  const int wpos = qp0 + 32 * wave;
  const int my_qpos = wpos + lr;
  const float sm_scale = 1.f / sqrtf((float)sh.hd);

  float qf[HDP / 2], dof[HDP / 2];
  load_reg_operand<HDP>(qf, qbase, rs, my_q, sh.T, sh.hd, hh, LOG2E * sm_scale);
  load_reg_operand<HDP>(dof, dobase, C, my_q, sh.T, sh.hd, hh, 1.f);
  float Dq;
  if (SEG) {
    Dq = my_q < sh.T ? Dws[(long long)bh * sh.T + my_q] : 0.f;
  } else {
    const float* obase = out + (long long)b * sh.T * C + (long long)h * sh.hd;
    float of[HDP / 2];
    load_reg_operand<HDP>(of, obase, C, my_q, sh.T, sh.hd, hh, 1.f);
    float part = 0.f;
#pragma unroll
    for (int s = 0; s < HDP / 2; ++s) part += dof[s] * of[s];
    Dq = part + __shfl_xor(part, 32, 64);
    if (hh == 0 && my_q < sh.T) Dws[(long long)bh * sh.T + my_q] = Dq;
  }
  const float lse2 = my_q < sh.T ? lse[(long long)bh * sh.T + my_q] * LOG2E : 0.f;

  floatx16 dq[HDP / 32];
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db) zero16(dq[db]);

  int nkb, n0;
  if (SEG) {
    n0 = seg_prefix_tiles(qp0 + 127, sg.k_pos[0], sg.seg);
    nkb = n0 + (Tk > sg.seg ? seg_prefix_tiles(qp0 + 127, sg.k_pos[1], sg.seg) : 0);
  } else {
    nkb = min(sh.T - 1, q0 + 127) / 32 + 1;
    n0 = nkb;
  }
  auto key_row = [&](int kb) { return SEG ? (kb < n0 ? 32 * kb : sg.seg + 32 * (kb - n0)) : 32 * kb; };
  auto key_pos = [&](int kb) { return SEG ? (kb < n0 ? sg.k_pos[0] + 32 * kb : sg.k_pos[1] + 32 * (kb - n0)) : 32 * kb; };

  floatx4 rk[HDP / 32], rv[HDP / 32];
  if (nkb > 0) {
    load_rows_clamped<HDP>(rk, kbase, ks, key_row(0), Tk, sh.hd, tid);
    load_rows_clamped<HDP>(rv, vbase, ks, key_row(0), Tk, sh.hd, tid);
    store_rows_masked<HDP, LDK>(smem, rk, tid, key_row(0), Tk, sh.hd);
    store_rows_masked<HDP, LDV>(smem + KSZ, rv, tid, key_row(0), Tk, sh.hd);
  }
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) {
      load_rows_clamped<HDP>(rk, kbase, ks, key_row(kb + 1), Tk, sh.hd, tid);
      load_rows_clamped<HDP>(rv, vbase, ks, key_row(kb + 1), Tk, sh.hd, tid);
    }
    const int kp0 = key_pos(kb);
    if (kp0 <= wpos + 31) {
      const float* sK = smem + cur * (KSZ + VSZ);
      const float* sV = sK + KSZ;
      floatx16 s, dp;
      zero16(s);
      zero16(dp);
      mma_rows_by_reg<HDP, LDK>(s, sK, qf, lr, hh);    // S^T  [key][q]
      mma_rows_by_reg<HDP, LDV>(dp, sV, dof, lr, hh);  // dP^T [key][q]
      const int kr0 = key_row(kb);
      if ((kp0 + 31 > wpos) || (kr0 + 32 > Tk)) {  // diagonal or ragged tile (uniform)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kk = acc_row(r, hh);
          const bool dead = (kp0 + kk > my_qpos) | (kr0 + kk >= Tk);
          const float p = dead ? 0.f : exp2_hw(s[r] - lse2);
          s[r] = p * (dp[r] - Dq);  // dS^T
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = exp2_hw(s[r] - lse2) * (dp[r] - Dq);
      }
      mma_tile_T_by_acc<HDP, LDK>(dq, sK, s, lr, hh);  // dQ^T[d][q] += K^T dS^T
    }
    if (more) {
      float* sN = smem + (cur ^ 1) * (KSZ + VSZ);
      store_rows_masked<HDP, LDK>(sN, rk, tid, key_row(kb + 1), Tk, sh.hd);
      store_rows_masked<HDP, LDV>(sN + KSZ, rv, tid, key_row(kb + 1), Tk, sh.hd);
    }
    __syncthreads();
  }
  float* stage = smem + wave * 32 * (HDP + 4);
  float* dqbase = dqkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  store_T_tile<HDP>(stage, dq, sm_scale, dqbase, rs, qw0, sh.T, sh.hd, lane,
                    SEG && (sg.flags & SEG_ACC_DQ));
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
// SEG: keys and values from sg.kv, dK/dV to sg.dkv (optionally added), queries
// visible by segment positions; dS ([B, H, T, Tk]) when positions are
// multiples of 128 (the segmented dQ product's tiles).
template <int HDP, bool SEG>
__global__ void __launch_bounds__(256, HDP <= 64 ? 2 : 1) attn_bwd_dkv_kernel(
    const float* __restrict__ dout, const float* __restrict__ qkv, const float* __restrict__ lse,
    const float* __restrict__ Dws, float* __restrict__ dqkv, float* __restrict__ dS, AttnShape sh,
    AttnSegs sg) {
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
  const int Tk = SEG ? sg.Tk : sh.T;
  const long long ks = SEG ? sg.kv_stride : rs;
  const float* qbase = qkv + (long long)b * sh.T * rs + (long long)h * sh.hd;
  const float* kbase = SEG ? sg.kv + (long long)b * Tk * ks + (long long)h * sh.hd : qbase + C;
  const float* vbase = kbase + C;
  const float* dobase = dout + (long long)b * sh.T * C + (long long)h * sh.hd;
  const float* lrow = lse + (long long)bh * sh.T;
  const float* drow = Dws + (long long)bh * sh.T;

  const int k0 = kt * 128;
  const int kw0 = k0 + 32 * wave;
  const int my_k = kw0 + lr;
  const int kp0 = SEG ? seg_pos(sg.k_pos, sg.seg, k0) : k0;  // the block's rows lie in one segment
  const int kwpos = kp0 + 32 * wave;
  const int my_kpos = kwpos + lr;
  const float sm_scale = 1.f / sqrtf((float)sh.hd);
  // dS / sqrt(hd) for the dQ product, [B, H, T, Tk]: this (b, h)'s rows, and
  // the byte offset of this lane's first element in a query tile (row 4 hh,
  // column my_k); register r of the tile is a scalar offset further.
  float* const ds_bh = dS ? dS + (long long)bh * sh.T * Tk : nullptr;
  const bool ds_lane = my_k < Tk;
  const unsigned ds_voff = 4u * (unsigned)(4 * hh * Tk + my_k);

  float kf[HDP / 2], vf[HDP / 2];
  load_reg_operand<HDP>(kf, kbase, ks, my_k, Tk, sh.hd, hh, LOG2E * sm_scale);
  load_reg_operand<HDP>(vf, vbase, ks, my_k, Tk, sh.hd, hh, 1.f);

  floatx16 dk[HDP / 32], dv[HDP / 32];
#pragma unroll
  for (int db = 0; db < HDP / 32; ++db) {
    zero16(dk[db]);
    zero16(dv[db]);
  }

  // streamed query tiles: causal, rows from the key tile's diagonal to the
  // end; SEG, a suffix of each query segment (c0 tiles of the first, from m0)
  int qb0, nq, c0, m1 = 0;
  if (SEG) {
    const int per = sg.seg / 32;
    qb0 = min(per, seg_suffix_first(kp0, sg.q_pos[0]));
    c0 = per - qb0;
    nq = c0;
    if (sh.T > sg.seg) {
      m1 = min(per, seg_suffix_first(kp0, sg.q_pos[1]));
      nq += per - m1;
    }
  } else {
    qb0 = k0 / 32;
    nq = max(0, (sh.T + 31) / 32 - qb0);
    c0 = nq;
  }
  auto q_row = [&](int j) { return SEG ? (j < c0 ? 32 * (qb0 + j) : sg.seg + 32 * (m1 + j - c0)) : 32 * (qb0 + j); };
  auto q_pos = [&](int j) {
    return SEG ? (j < c0 ? sg.q_pos[0] + 32 * (qb0 + j) : sg.q_pos[1] + 32 * (m1 + j - c0)) : 32 * (qb0 + j);
  };

  floatx4 rq[HDP / 32], rdo[HDP / 32];
  float rl = 0.f, rd = 0.f;
  auto load_q = [&](int j) {
    const int r0 = q_row(j);
    load_rows_clamped<HDP>(rq, qbase, rs, r0, sh.T, sh.hd, tid);
    load_rows_clamped<HDP>(rdo, dobase, C, r0, sh.T, sh.hd, tid);
    if (tid < 32) {
      const int t = min(r0 + tid, sh.T - 1);
      rl = lrow[t];
      rd = drow[t];
    }
  };
  auto store_q = [&](float* sb, int j) {
    const int r0 = q_row(j);
    store_rows_masked<HDP, LD>(sb, rq, tid, r0, sh.T, sh.hd);
    store_rows_masked<HDP, LD>(sb + TSZ, rdo, tid, r0, sh.T, sh.hd);
    if (tid < 32) {
      const bool ok = r0 + tid < sh.T;
      sb[2 * TSZ + tid] = ok ? rl * LOG2E : INFINITY;  // rows past T give P = 0
      sb[2 * TSZ + 32 + tid] = ok ? rd : 0.f;
    }
  };
  if (nq > 0) {
    load_q(0);
    store_q(smem, 0);
  }
  __syncthreads();

  for (int j = 0; j < nq; ++j) {
    const int cur = j & 1;
    const bool more = j + 1 < nq;
    if (more) load_q(j + 1);
    const int qv0 = q_row(j);   // first row of the query tile
    const int qp = q_pos(j);    // its first position
    const bool live = qp + 31 >= kwpos && kw0 < Tk;  // some query of the tile sees this wave's keys
    floatx16 dp;
    if (live) {
      const float* sQ = smem + cur * BUF;
      const float* sdO = sQ + TSZ;
      const float* sl = sQ + 2 * TSZ;
      const float* sd = sl + 32;
      floatx16 s;
      zero16(s);
      zero16(dp);
      mma_rows_by_reg<HDP, LD>(s, sQ, kf, lr, hh);    // S  [q][key]
      mma_rows_by_reg<HDP, LD>(dp, sdO, vf, lr, hh);  // dP [q][key]
      // P needs only S: it is formed while the dP products run, and the dV
      // products (which need only P) run while dS is formed.
      if ((qp < kwpos + 31) || (kw0 + 32 > Tk)) {  // diagonal or ragged tile (uniform)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int qi = acc_row(r, hh);
          const bool dead = (my_kpos > qp + qi) | (my_k >= Tk);
          s[r] = dead ? 0.f : exp2_hw(s[r] - sl[qi]);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = exp2_hw(s[r] - sl[acc_row(r, hh)]);
      }
      mma_tile_T_by_acc<HDP, LD>(dv, sdO, s, lr, hh);  // dV^T[d][key] += dO^T P
#pragma unroll
      for (int r = 0; r < 16; ++r) dp[r] = s[r] * (dp[r] - sd[acc_row(r, hh)]);  // dS
      mma_tile_T_by_acc<HDP, LD>(dk, sQ, dp, lr, hh);  // dK^T[d][key] += Q^T dS
    }
    // The next tile goes to LDS before this tile's dS is stored: loads and
    // stores retire in order on one counter, so a wait for the next tile's
    // loads issued after the stores would also wait for the stores to be
    // written.
    if (more) store_q(smem + (cur ^ 1) * BUF, j + 1);
    if (ds_bh && ds_lane && (live || qp < kwpos)) {
      // One buffer resource per query tile, limited to the tile's rows below
      // T: the stores of rows past T fall outside it and are dropped.  The
      // tile base and the per-register offsets are scalars, so the 16
      // stores need no vector address arithmetic.  Query tiles of the
      // diagonal 128-row tile that precede this wave's keys are fully masked
      // and stored as zeros, because the dQ product of that tile sums keys
      // up to the tile's end.
      const auto rs = __builtin_amdgcn_make_buffer_rsrc(ds_bh + (long long)qv0 * Tk, (short)0,
                                                        4 * Tk * min(32, sh.T - qv0), 0x00020000);
#pragma unroll
      for (int r = 0; r < 16; ++r)
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, live ? dp[r] * sm_scale : 0.f), rs,
                                              ds_voff, 4 * Tk * (8 * (r >> 2) + (r & 3)), 0);
    }
    __syncthreads();
  }
  float* stage = smem + wave * 32 * (HDP + 4);
  float* dkbase = SEG ? sg.dkv + (long long)b * Tk * ks + (long long)h * sh.hd
                      : dqkv + (long long)b * sh.T * rs + (long long)h * sh.hd + C;
  const bool add = SEG && (sg.flags & SEG_ACC_DKV);
  store_T_tile<HDP>(stage, dk, sm_scale, dkbase, ks, kw0, Tk, sh.hd, lane, add);
  __syncthreads();
  store_T_tile<HDP>(stage, dv, 1.f, dkbase + C, ks, kw0, Tk, sh.hd, lane, add);
}

bt_status check_attn(const void* a, const void* b2, int B, int T, int H, int hd, const char* who) {
  BT_RETURN_IF(B < 1 || T < 1 || H < 1, BT_ESHAPE, "%s: B=%d T=%d H=%d must be >= 1", who, B, T, H);
  BT_RETURN_IF(hd < 4 || hd > 128 || (hd & 3), BT_ESHAPE,
               "%s: head dim %d unsupported (multiple of 4, <= 128)", who, hd);
  BT_RETURN_IF(!a || !b2, BT_EINVAL, "%s: NULL pointer", who);
  BT_RETURN_IF((long long)B * H * ((T + 127) / 128) > 0x7fffffffLL, BT_ESHAPE, "%s: grid too large", who);
  return BT_OK;
}

// Kernel launches by padded head dim.
template <bool SEG>
void launch_fwd(int hd, dim3 grid, hipStream_t s, const float* qkv, float* out, float* lse,
                const AttnShape& sh, const AttnSegs& sg) {
  if (hd <= 32)
    hipLaunchKernelGGL((attn_fwd_kernel<32, SEG>), grid, dim3(256), 0, s, qkv, out, lse, sh, sg);
  else if (hd <= 64) {
    // direct-to-LDS key / value tiles when every key tile is full and the
    // per-lane copy offsets (32 rows of the token stride) fit in 32 bits
    if (!SEG && hd == 64 && sh.T % 32 == 0 && sh.row_stride < (1LL << 24))
      hipLaunchKernelGGL((attn_fwd_kernel<64, false, true>), grid, dim3(256), 0, s, qkv, out, lse, sh, sg);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<64, SEG>), grid, dim3(256), 0, s, qkv, out, lse, sh, sg);
  }
  else
    hipLaunchKernelGGL((attn_fwd_kernel<128, SEG>), grid, dim3(256), 0, s, qkv, out, lse, sh, sg);
}

template <bool SEG>
void launch_dq(int hd, dim3 grid, hipStream_t s, const float* dout, const float* qkv, const float* out,
               const float* lse, float* dqkv, float* D, const AttnShape& sh, const AttnSegs& sg) {
  if (hd <= 32)
    hipLaunchKernelGGL((attn_bwd_dq_kernel<32, SEG>), grid, dim3(256), 0, s, dout, qkv, out, lse, dqkv, D, sh, sg);
  else if (hd <= 64)
    hipLaunchKernelGGL((attn_bwd_dq_kernel<64, SEG>), grid, dim3(256), 0, s, dout, qkv, out, lse, dqkv, D, sh, sg);
  else
    hipLaunchKernelGGL((attn_bwd_dq_kernel<128, SEG>), grid, dim3(256), 0, s, dout, qkv, out, lse, dqkv, D, sh, sg);
}

template <bool SEG>
void launch_dkv(int hd, dim3 grid, hipStream_t s, const float* dout, const float* qkv, const float* lse,
                const float* D, float* dqkv, float* dS, const AttnShape& sh, const AttnSegs& sg) {
  if (hd <= 32)
    hipLaunchKernelGGL((attn_bwd_dkv_kernel<32, SEG>), grid, dim3(256), 0, s, dout, qkv, lse, D, dqkv, dS, sh, sg);
  else if (hd <= 64)
    hipLaunchKernelGGL((attn_bwd_dkv_kernel<64, SEG>), grid, dim3(256), 0, s, dout, qkv, lse, D, dqkv, dS, sh, sg);
  else
    hipLaunchKernelGGL((attn_bwd_dkv_kernel<128, SEG>), grid, dim3(256), 0, s, dout, qkv, lse, D, dqkv, dS, sh, sg);
}

bt_status launch_d(const float* dout, const float* out, float* D, int B, int T, int H, int hd, hipStream_t s) {
  const long long rows = (long long)B * T;
  const unsigned gd = (unsigned)(rows < 8192 ? rows : 8192);
  const size_t part_bytes = (size_t)H * hd / 4 * sizeof(float);
  BT_RETURN_IF(part_bytes > 64 * 1024, BT_ESHAPE, "attention backward: H * hd = %d too large", H * hd);
  hipLaunchKernelGGL(attn_bwd_d_kernel, dim3(gd), dim3(256), part_bytes, s, dout, out, D, B, T, H, hd);
  return check_launch("attn_bwd_d_kernel");
}

// Validates a rank's segment description and fills the kernel's copy.
bt_status make_segs(const bt_cp_segments* g, int H, int hd, const float* kv, float* dkv, long long kv_stride,
                    AttnSegs* sg, int* Tq, const char* who) {
  BT_RETURN_IF(!g, BT_EINVAL, "%s: segments are NULL", who);
  BT_RETURN_IF(g->seg < 128 || g->seg % 128, BT_ESHAPE, "%s: segment length %d must be a positive multiple of 128",
               who, g->seg);
  BT_RETURN_IF(g->n_q < 1 || g->n_q > 2 || g->n_k < 1 || g->n_k > 2, BT_ESHAPE,
               "%s: 1 or 2 segments per side (got %d, %d)", who, g->n_q, g->n_k);
  for (int i = 0; i < 2; ++i) {
    const bool q_used = i < g->n_q, k_used = i < g->n_k;
    BT_RETURN_IF(q_used && (g->q_pos[i] < 0 || g->q_pos[i] % 32), BT_ESHAPE,
                 "%s: query segment position %d must be a non-negative multiple of 32", who, g->q_pos[i]);
    BT_RETURN_IF(k_used && (g->k_pos[i] < 0 || g->k_pos[i] % 32), BT_ESHAPE,
                 "%s: key segment position %d must be a non-negative multiple of 32", who, g->k_pos[i]);
    BT_RETURN_IF((q_used && g->q_pos[i] > 0x7fffffff - g->seg) || (k_used && g->k_pos[i] > 0x7fffffff - g->seg),
                 BT_ESHAPE, "%s: positions overflow", who);
  }
  BT_RETURN_IF(!kv, BT_EINVAL, "%s: kv is NULL", who);
  BT_RETURN_IF(!aligned16(kv) || (dkv && !aligned16(dkv)), BT_EALIGN, "%s: kv/dkv must be 16-byte aligned", who);
  BT_RETURN_IF(kv_stride < 2LL * H * hd || (kv_stride & 3), BT_ESHAPE,
               "%s: kv token stride %lld must be a multiple of 4 and >= 2 H hd = %d", who, kv_stride, 2 * H * hd);
  *sg = AttnSegs{};
  sg->kv = kv;
  sg->dkv = dkv;
  sg->kv_stride = kv_stride;
  sg->seg = g->seg;
  sg->Tk = g->n_k * g->seg;
  for (int i = 0; i < 2; ++i) {
    sg->q_pos[i] = i < g->n_q ? g->q_pos[i] : 0;
    sg->k_pos[i] = i < g->n_k ? g->k_pos[i] : 0;
  }
  *Tq = g->n_q * g->seg;
  return BT_OK;
}

__global__ void __launch_bounds__(256) lse_merge_kernel(float* __restrict__ out, float* __restrict__ lse,
                                                        const float* __restrict__ bout,
                                                        const float* __restrict__ blse, int B, int T, int H,
                                                        int hd) {
  // 64 rows (b, t, h) per pass: 64 lanes take the rows' weights, then the
  // block streams the rows' contiguous 64 hd floats of out.
  __shared__ float w[64];
  const long long rows = (long long)B * T * H;
  const int q4 = hd / 4;
  for (long long r0 = (long long)blockIdx.x * 64; r0 < rows; r0 += (long long)gridDim.x * 64) {
    if (threadIdx.x < 64) {
      const long long r = r0 + threadIdx.x;
      float wt = MERGE_KEEP;
      if (r < rows) {
        const int h = (int)(r % H);
        const long long bt = r / H;
        const long long li = ((bt / T) * H + h) * T + bt % T;
        float nl;
        wt = lse_merge_row(lse[li], blse[li], &nl);
        lse[li] = nl;
      }
      w[threadIdx.x] = wt;
    }
    __syncthreads();
    const long long nrow = rows - r0 < 64 ? rows - r0 : 64;
    const long long n4 = nrow * q4;
    floatx4* o4 = reinterpret_cast<floatx4*>(out + r0 * hd);
    const floatx4* b4 = reinterpret_cast<const floatx4*>(bout + r0 * hd);
    for (long long i = threadIdx.x; i < n4; i += 256) {
      const float wt = w[i / q4];
      if (wt != MERGE_KEEP) o4[i] = lse_merge_apply(wt, wt == MERGE_TAKE ? b4[i] : o4[i], b4[i]);
    }
    __syncthreads();
  }
}

__global__ void cp_shard_tokens_kernel(const int32_t* __restrict__ tokens, int32_t* __restrict__ local, int B,
                                       int T, int seg, int c0, int c1) {
  const long long n = (long long)B * 2 * seg;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
    const long long b = i / (2 * seg);
    const int j = (int)(i % (2 * seg));
    const int pos = j < seg ? c0 * seg + j : c1 * seg + (j - seg);
    local[i] = tokens[b * T + pos];
  }
}

}  // namespace
}  // namespace bt

using namespace bt;

extern "C" bt_status bt_attention_fwd(const float* qkv, float* out, float* lse, int B, int T, int H,
                                      int hd, void* stream) {
  bt::clear_error();
  BT_TRY(check_attn(qkv, out, B, T, H, hd, "bt_attention_fwd"));
  BT_RETURN_IF(!lse, BT_EINVAL, "bt_attention_fwd: lse is NULL");
  BT_RETURN_IF(!aligned16(qkv) || !aligned16(out), BT_EALIGN, "bt_attention_fwd: qkv/out must be 16-byte aligned");
  AttnShape sh{B, T, H, hd, 3LL * H * hd};
  dim3 grid((unsigned)(B * H * ((T + 127) / 128)));
  launch_fwd<false>(hd, grid, as_stream(stream), qkv, out, lse, sh, AttnSegs{});
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
  bt::clear_error();
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
    BT_TRY(launch_d(dout, out, D, B, T, H, hd, s));
    launch_dkv<false>(hd, gq, s, dout, qkv, lse, D, dqkv, dS, sh, AttnSegs{});
    BT_TRY(check_launch("attn_bwd_dkv_kernel"));
    const long long rs = sh.row_stride;
    // per (b, h): dQ [T][hd] (rows of dqkv, stride 3 H hd) = dS [T][T] K [T][hd]
    return gemm_causal_batched(T, hd, T, dS, T, (long long)H * T * T, (long long)T * T,
                               qkv + (long long)H * hd, (int)rs, (long long)T * rs, hd,
                               dqkv, (int)rs, (long long)T * rs, hd, B, H, s);
  }
  launch_dq<false>(hd, gq, s, dout, qkv, out, lse, dqkv, D, sh, AttnSegs{});
  BT_TRY(check_launch("attn_bwd_dq_kernel"));
  launch_dkv<false>(hd, gq, s, dout, qkv, lse, D, dqkv, nullptr, sh, AttnSegs{});
  return check_launch("attn_bwd_dkv_kernel");
}

// ---------------------------------------------------------------- context parallelism

extern "C" bt_status bt_cp_rank_segments(int T, int W, int rank, int shard, bt_cp_segments* out) {
  bt::clear_error();
  BT_RETURN_IF(!out, BT_EINVAL, "bt_cp_rank_segments: out is NULL");
  BT_RETURN_IF(W < 1 || rank < 0 || rank >= W || shard < 0 || shard >= W, BT_EINVAL,
               "bt_cp_rank_segments: rank %d / shard %d outside [0, W=%d)", rank, shard, W);
  BT_RETURN_IF(T < 1 || T % (2 * W * 128), BT_ESHAPE,
               "bt_cp_rank_segments: T=%d must be a multiple of 2 W 128 = %d", T, 2 * W * 128);
  const int seg = T / (2 * W);
  out->seg = seg;
  out->n_q = out->n_k = 2;
  out->q_pos[0] = rank * seg;
  out->q_pos[1] = (2 * W - 1 - rank) * seg;
  out->k_pos[0] = shard * seg;
  out->k_pos[1] = (2 * W - 1 - shard) * seg;
  return BT_OK;
}

extern "C" bt_status bt_cp_shard_tokens(const int32_t* tokens, int32_t* local, int B, int T, int W, int rank,
                                        void* stream) {
  bt::clear_error();
  bt_cp_segments g;
  BT_TRY(bt_cp_rank_segments(T, W, rank, rank, &g));
  BT_RETURN_IF(B < 1, BT_ESHAPE, "bt_cp_shard_tokens: B=%d", B);
  BT_RETURN_IF(!tokens || !local, BT_EINVAL, "bt_cp_shard_tokens: NULL pointer");
  BT_RETURN_IF((long long)B * T > 0x7fffffffLL, BT_ESHAPE, "bt_cp_shard_tokens: too many tokens");
  const long long n = (long long)B * 2 * g.seg;
  const unsigned grid = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(cp_shard_tokens_kernel, dim3(grid), dim3(256), 0, as_stream(stream), tokens, local, B, T,
                     g.seg, rank, 2 * W - 1 - rank);
  return check_launch("cp_shard_tokens_kernel");
}

extern "C" bt_status bt_attention_block_fwd(const float* qkv, const float* kv, long long kv_stride, float* out,
                                            float* lse, int merge, int B, int H, int hd,
                                            const bt_cp_segments* segs, void* stream) {
  bt::clear_error();
  AttnSegs sg;
  int Tq = 0;
  BT_TRY(make_segs(segs, H, hd, kv, nullptr, kv_stride, &sg, &Tq, "bt_attention_block_fwd"));
  BT_TRY(check_attn(qkv, out, B, Tq, H, hd, "bt_attention_block_fwd"));
  BT_RETURN_IF(!lse, BT_EINVAL, "bt_attention_block_fwd: lse is NULL");
  BT_RETURN_IF(!aligned16(qkv) || !aligned16(out), BT_EALIGN,
               "bt_attention_block_fwd: qkv/out must be 16-byte aligned");
  BT_RETURN_IF(merge != 0 && merge != 1, BT_EINVAL, "bt_attention_block_fwd: merge must be 0 or 1");
  sg.flags = merge ? SEG_MERGE : 0;
  AttnShape sh{B, Tq, H, hd, 3LL * H * hd};
  launch_fwd<true>(hd, dim3((unsigned)(B * H * (Tq / 128))), as_stream(stream), qkv, out, lse, sh, sg);
  return check_launch("attn_fwd_kernel (block)");
}

extern "C" bt_status bt_attention_lse_merge(float* out, float* lse, const float* block_out, const float* block_lse,
                                            int B, int T, int H, int hd, void* stream) {
  bt::clear_error();
  BT_RETURN_IF(B < 1 || T < 1 || H < 1 || hd < 4 || (hd & 3), BT_ESHAPE,
               "bt_attention_lse_merge: bad shape B=%d T=%d H=%d hd=%d", B, T, H, hd);
  BT_RETURN_IF(!out || !lse || !block_out || !block_lse, BT_EINVAL, "bt_attention_lse_merge: NULL pointer");
  BT_RETURN_IF(!aligned16(out) || !aligned16(block_out), BT_EALIGN,
               "bt_attention_lse_merge: out/block_out must be 16-byte aligned");
  const long long rows = (long long)B * T * H;
  const long long blocks = (rows + 63) / 64;
  const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
  hipLaunchKernelGGL(lse_merge_kernel, dim3(grid), dim3(256), 0, as_stream(stream), out, lse, block_out, block_lse,
                     B, T, H, hd);
  return check_launch("lse_merge_kernel");
}

extern "C" bt_status bt_attention_rowdot(const float* dout, const float* out, float* D, int B, int T, int H, int hd,
                                         void* stream) {
  bt::clear_error();
  BT_TRY(check_attn(dout, out, B, T, H, hd, "bt_attention_rowdot"));
  BT_RETURN_IF(!D, BT_EINVAL, "bt_attention_rowdot: D is NULL");
  BT_RETURN_IF(!aligned16(dout) || !aligned16(out), BT_EALIGN,
               "bt_attention_rowdot: dout/out must be 16-byte aligned");
  return launch_d(dout, out, D, B, T, H, hd, as_stream(stream));
}

// The stored-dS method of a ring step: needs positions that are multiples of
// 128 (the dQ product's row tiles then meet the key tiles on their edges).
static bool block_stores_ds(const bt_cp_segments* g) {
  for (int i = 0; i < g->n_q; ++i)
    if (g->q_pos[i] % 128) return false;
  for (int i = 0; i < g->n_k; ++i)
    if (g->k_pos[i] % 128) return false;
  return true;
}

extern "C" size_t bt_attention_block_bwd_ws_bytes(int B, int H, int hd, const bt_cp_segments* segs) {
  (void)hd;
  if (!segs || B <= 0 || H <= 0 || segs->seg <= 0 || segs->n_q < 1 || segs->n_q > 2 || segs->n_k < 1 ||
      segs->n_k > 2 || !block_stores_ds(segs))
    return 0;
  return align_up((size_t)B * H * segs->n_q * segs->seg * segs->n_k * segs->seg * sizeof(float), 256);
}

extern "C" bt_status bt_attention_block_bwd(const float* dout, const float* qkv, const float* kv, long long kv_stride,
                                            const float* lse, const float* D, float* dqkv, float* dkv,
                                            int accumulate, void* ws, size_t ws_bytes, int B, int H, int hd,
                                            const bt_cp_segments* segs, void* stream) {
  bt::clear_error();
  AttnSegs sg;
  int Tq = 0;
  BT_TRY(make_segs(segs, H, hd, kv, dkv, kv_stride, &sg, &Tq, "bt_attention_block_bwd"));
  BT_TRY(check_attn(qkv, dout, B, Tq, H, hd, "bt_attention_block_bwd"));
  BT_TRY(check_attn(kv, dout, B, sg.Tk, H, hd, "bt_attention_block_bwd"));
  BT_RETURN_IF(!lse || !D || !dqkv || !dkv, BT_EINVAL, "bt_attention_block_bwd: NULL pointer");
  BT_RETURN_IF(!aligned16(qkv) || !aligned16(dout) || !aligned16(dqkv) || (ws && !aligned16(ws)), BT_EALIGN,
               "bt_attention_block_bwd: tensors and workspace must be 16-byte aligned");
  BT_RETURN_IF(accumulate < 0 || accumulate > 3, BT_EINVAL, "bt_attention_block_bwd: accumulate must be 0..3");
  BT_RETURN_IF(dqkv == qkv || dkv == kv, BT_EINVAL, "bt_attention_block_bwd: gradients must not alias inputs");
  sg.flags = accumulate;
  AttnShape sh{B, Tq, H, hd, 3LL * H * hd};
  hipStream_t s = as_stream(stream);
  const size_t need = bt_attention_block_bwd_ws_bytes(B, H, hd, segs);
  const dim3 gk((unsigned)(B * H * (sg.Tk / 128)));
  if (need && ws && ws_bytes >= need) {
    // key-major pass with dS stored, then dQ (+)= dS K over the visible key
    // ranges of each 128-row tile on the matrix-core GEMM
    float* dS = static_cast<float*>(ws);
    launch_dkv<true>(hd, gk, s, dout, qkv, lse, D, nullptr, dS, sh, sg);
    BT_TRY(check_launch("attn_bwd_dkv_kernel (block, dS)"));
    const long long rs = sh.row_stride, ks = kv_stride, Tk = sg.Tk;
    return gemm_segmented_batched(Tq, hd, sg.Tk, dS, sg.Tk, (long long)H * Tq * Tk, (long long)Tq * Tk, kv, (int)ks,
                                  Tk * ks, hd, dqkv, (int)rs, (long long)Tq * rs, hd, B, H,
                                  (accumulate & SEG_ACC_DQ) ? 1.f : 0.f, sg.seg, sg.q_pos, sg.k_pos, s);
  }
  launch_dq<true>(hd, dim3((unsigned)(B * H * (Tq / 128))), s, dout, qkv, nullptr, lse, dqkv,
                  const_cast<float*>(D), sh, sg);
  BT_TRY(check_launch("attn_bwd_dq_kernel (block)"));
  launch_dkv<true>(hd, gk, s, dout, qkv, lse, D, nullptr, nullptr, sh, sg);
  return check_launch("attn_bwd_dkv_kernel (block)");
}
