// FP32 GEMM family on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Serves every dense projection of the training step in its three layouts
// (native GEMM library paragraph of "Implementation": QKV, attention-output
// and MLP projections in forward and backward layouts, plus the tied LM
// head):  forward Y = X W (NN), input gradient dX = dY W^T (NT), weight
// gradient dW = X^T dY (TN, reduction over tokens, split along K).
//
// Design (gfx950):
//  * block tile 128 x 128 x BK (BK = 16 at 4 blocks per CU, or BK = 32 at 2),
//    256 threads = 4 waves in a 2 x 2 grid, each wave owns a 64 x 64 sub-tile
//    = 2 x 2 MFMA 32x32 accumulators (64 VGPRs).  The kernel is written for
//    any WM x WN wave grid; 256 x 128, 128 x 256 and 256 x 256 block tiles are
//    not launched: on MI355X they gain up to 6% on plain products with
//    thousands of tiles but lose 10-35% on the 768-column products and the
//    epilogue products, so the model's step is slower with them.
//  * when every tile of a launch is full (M, N multiples of 128, K range a
//    multiple of BK: all GPT-2 shapes) operand tiles go straight from global
//    memory into LDS (global_load_lds_dwordx4, 1 KB per wave instruction):
//    no staging VGPRs, no LDS store instructions.  Ragged shapes stage them
//    global -> VGPR -> LDS with bounds checks.  On MI355X the direct copies
//    raised the matrix-pipe busy fraction of the NN / TN products by 3-5
//    points (measured with SQ_VALU_MFMA_BUSY_CYCLES).  Their addresses are
//    a wave-uniform tile base in SGPRs plus a fixed per-lane 32-bit offset,
//    and the LDS destinations are scalar too, so the k-loop spends no vector
//    instruction on them: a vector instruction a wave issues between its
//    MFMAs delays them (4-8 cycles each on MI355X), and moving the 64-bit
//    address arithmetic and readfirstlanes to the scalar unit made the
//    step's products 4-10% faster.
//  * LDS layouts follow the source layout: K-contiguous rows [rows][BK] with
//    an XOR swizzle of 16-byte chunks; MN-contiguous rows [BK][128] with the
//    32-column halves swapped in every other group of 8 k-rows (direct copy)
//    or padded to [BK][132] (staged).  Two LDS buffers, one barrier per
//    k-tile, the next tile in flight while the MFMAs run, wave priority
//    raised while a wave issues MFMAs.
//  * the MFMA k-slot of lane half h at step s is k = 8h + (s mod 8) +
//    16 (s div 8) (s < BK/2): K-contiguous tiles are read as float4 (4 steps
//    at once), MN-contiguous tiles as b32 with the two lane halves 8 rows
//    apart; both reads are free of LDS bank conflicts.
//  * blocks are remapped so that each XCD (round-robin dispatch over 8 XCDs,
//    one L2 each) receives a contiguous range of a grouped (8 tile-rows)
//    tile order, so concurrently running tiles share A rows / B columns in L2.
//  * low-parallelism weight-gradient shapes (small M x N, long K) are split
//    along K; partials go to a workspace and are summed in a fixed order.
//    Tile depth and split count are chosen per shape from a model of how
//    the blocks land on the 256 CUs (blocks per CU, resident blocks).
//  * fused epilogues: bias, bias + tanh-GELU (optionally storing the
//    pre-activation), GELU-backward (multiply by gelu'(pre)), residual add and
//    beta = 1 accumulation.
//  * the weight-gradient product can also return the column sums of dY (the
//    bias gradient) from the B data it already reads, so the bias gradient
//    costs no extra pass over dY.
#include <mutex>

#include "bt_internal.h"

namespace bt {
namespace {

constexpr int NUM_CU = 256;
constexpr size_t MAX_SPLIT_WS = (size_t)1 << 30;  // largest split-K partial buffer considered

struct GemmParams {
  const float* A;
  const float* B;
  float* C;
  const float* bias;
  float* preact;
  const float* gelu_in;
  const float* residual;
  float* ws;
  float* colsum;     // optional column sums of op(B) over K (bias gradient of a weight-gradient product)
  float* ws_colsum;  // split-K partial column sums [splits][N]
  long long lda, ldb, ldc;
  int M, N, K;
  int ksplit;   // K range handled by one split (multiple of BK)
  int splits;
  int tiles_m, tiles_n;
  float beta;
  // batched products only: batch y addresses A + (y / batch_h) sa_b +
  // (y % batch_h) sa_h (likewise B, C)
  int nbatch, batch_h;
  long long sa_b, sa_h, sb_b, sb_h, sc_b, sc_h;
  // segmented batched products only: rows of A (and C) are 1 or 2 segments
  // of `seg` rows starting at positions q_pos[i], the K range 1 or 2 such
  // segments at k_pos[i]; output row i sums the k whose position is at most
  // the last position of its BM-row tile
  int seg;
  int q_pos[2], k_pos[2];
};

// LDS floats of one R-row operand tile: K-contiguous [R][BK] (swizzled) or
// MN-contiguous [BK][R + 4] (the pad keeps the two lane halves, 8 k-rows
// apart, on different banks); MN-contiguous tiles copied directly into LDS
// are unpadded [BK][R] with an XOR swizzle instead.
template <bool KC, int R, int BK, bool DTL>
struct TileSize {
  static constexpr int value = KC ? R * BK : BK * (DTL ? R : R + 4);
};

// float4 registers per thread that stage one R-row operand tile
template <int R, int BK, int NT>
struct TileVecs {
  static constexpr int value = R * BK / (4 * NT);
  static_assert(value >= 1 && R * BK == value * 4 * NT, "tile does not divide over the block");
};

// K-contiguous tiles are stored unpadded ([rows][BK]) with the 16-byte chunk
// index of each row XORed by a few row bits: a b128 read of one chunk by 32
// consecutive rows spreads over all LDS banks without a pad column.
template <int BK>
__device__ __forceinline__ int kc_swizzle(int row) {
  return BK == 16 ? ((row >> 2) & 3) : ((row >> 1) & 7);
}

// Unpadded MN-contiguous tiles: in k-rows with bit 3 set the two 32-column
// halves of every 64-column group trade places, so a fragment read (lane
// halves 8 k-rows apart, 32 consecutive columns each) hits distinct banks.
__device__ __forceinline__ int mn_swizzle(int k) { return ((k >> 3) & 1) << 5; }


// Per-lane byte offsets of the NI direct copies (1 KB slices) a wave issues
// for one R x BK operand tile, relative to the tile's first element (row 0,
// k 0 of the tile): at most R rows (K-contiguous) or BK rows (MN-contiguous)
// of the operand, so 32 bits suffice for any leading dimension the ABI takes.
// The tile's base address is wave-uniform and lives in SGPRs; advancing it
// by a k-tile is one scalar add, and no vector instruction is spent on the
// copies in the k-loop.
template <bool KC, int R, int BK, int NI>
__device__ __forceinline__ void copy_offsets(unsigned (&o)[NI], long long ld, int wave, int lane) {
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int slice = wave * NI + j;
    if (KC) {
      constexpr int TPR = BK / 4, RPS = 64 / TPR;  // rows per 1 KB slice
      const int row = slice * RPS + lane / TPR;
      const int q = (lane % TPR) ^ kc_swizzle<BK>(row);
      o[j] = (unsigned)(((long long)row * ld + 4 * q) * 4);
    } else {
      constexpr int LPK = R / 4, KPS = 64 / LPK;  // lanes per k-row, k-rows per slice
      const int k = slice * KPS + lane / LPK;
      const int col = (4 * (lane % LPK)) ^ mn_swizzle(k);
      o[j] = (unsigned)(((long long)k * ld + col) * 4);
    }
  }
}

// The NI copies of one operand tile: `base` is the tile's first element
// (wave-uniform), `lds` the LDS byte address of this wave's first slice.
// The per-lane copy offsets are 32-bit: a tile spans at most 256 rows (or
// k-rows) of its operand, so leading dimensions below 2^22 floats keep every
// offset below 4 GiB.  Wider operands take the staged path (64-bit addresses).
inline bool copy_offsets_fit(long long lda, long long ldb) {
  return lda < (1LL << 22) && ldb < (1LL << 22);
}

template <int NI>
__device__ __forceinline__ void copy_issue(const float* base, const unsigned (&o)[NI], unsigned lds) {
#pragma unroll
  for (int j = 0; j < NI; ++j) copy16_to_lds_sbase(base, o[j], lds + 1024u * j);
}

// Global -> register staging of one R x BK operand tile (NV float4 per
// thread).  rows = M (or N) extent, kbeg/kend = k range of this split.
template <bool KC, int R, int BK, int NT, int NV = TileVecs<R, BK, NT>::value>
__device__ __forceinline__ void load_tile(floatx4 (&r)[NV], const float* __restrict__ X, long long ld,
                                          int row0, int rows, int k0, int kend, int tid) {
  if (KC) {
    // [rows][K]: BK/4 threads per row, 4 consecutive k each (BK*4 bytes per row)
    constexpr int TPR = BK / 4, RPP = NT / TPR;
    const int kk = k0 + 4 * (tid % TPR);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int row = row0 + tid / TPR + RPP * i;
      if (row < rows && kk < kend)
        r[i] = *reinterpret_cast<const floatx4*>(X + (long long)row * ld + kk);
      else
        r[i] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
  } else {
    // [K][rows]: R/4 threads per k row, thread -> (k = tid / TPK + KPP i, col = 4 (tid % TPK))
    constexpr int TPK = R / 4, KPP = NT / TPK;
    const int col = row0 + 4 * (tid % TPK);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int kk = k0 + tid / TPK + KPP * i;
      if (kk < kend && col < rows)
        r[i] = *reinterpret_cast<const floatx4*>(X + (long long)kk * ld + col);
      else
        r[i] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
  }
}

template <bool KC, int R, int BK, int NT, int NV = TileVecs<R, BK, NT>::value>
__device__ __forceinline__ void store_tile(float* __restrict__ s, const floatx4 (&r)[NV], int tid) {
  if (KC) {
    constexpr int TPR = BK / 4, RPP = NT / TPR;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int row = tid / TPR + RPP * i;
      *reinterpret_cast<floatx4*>(s + row * BK + 4 * ((tid % TPR) ^ kc_swizzle<BK>(row))) = r[i];
    }
  } else {
    constexpr int TPK = R / 4, KPP = NT / TPK;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      *reinterpret_cast<floatx4*>(s + (tid / TPK + KPP * i) * (R + 4) + 4 * (tid % TPK)) = r[i];
  }
}

// Fragment for 4 consecutive MFMA steps (chunk c) of one 32-row block.
template <bool KC, int R, int BK, bool DTL>
__device__ __forceinline__ floatx4 read_frag(const float* __restrict__ s, int row, int koff) {
  constexpr int LDM = DTL ? R : R + 4;
  if (!KC && DTL) {
    floatx4 v;
    v[0] = s[(koff + 0) * LDM + (row ^ mn_swizzle(koff + 0))];
    v[1] = s[(koff + 1) * LDM + (row ^ mn_swizzle(koff + 1))];
    v[2] = s[(koff + 2) * LDM + (row ^ mn_swizzle(koff + 2))];
    v[3] = s[(koff + 3) * LDM + (row ^ mn_swizzle(koff + 3))];
    return v;
  }
  if (KC) {
    return *reinterpret_cast<const floatx4*>(s + row * BK + 4 * ((koff >> 2) ^ kc_swizzle<BK>(row)));
  } else {
    floatx4 v;
    v[0] = s[(koff + 0) * LDM + row];
    v[1] = s[(koff + 1) * LDM + row];
    v[2] = s[(koff + 2) * LDM + row];
    v[3] = s[(koff + 3) * LDM + row];
    return v;
  }
}

// Epilogue of one 32 x 32 accumulator block (register r of lane (lr, hh) is
// row i0 + 8 (r/4) + 4 hh + r%4, column j).  Every input the epilogue reads
// (bias, GELU pre-activation, residual, old C) is loaded before the first
// store: C may alias nothing, but the compiler cannot know that, and
// interleaved load/store pairs would serialise on memory latency.
template <int EPI>
__device__ __forceinline__ void epilogue_block(const GemmParams& p, const floatx16& acc, int i0, int j, int hh,
                                               float bj) {
  if (j >= p.N) return;
  const bool has_res = p.residual != nullptr;
  const bool has_old = p.beta != 0.f;
  constexpr int EC = 4;  // rows whose inputs are loaded together (8 or 16 spill at 4 waves per SIMD)
#pragma unroll
  for (int r0 = 0; r0 < 16; r0 += EC) {
    float gin[EC], res[EC], old[EC];
#pragma unroll
    for (int e = 0; e < EC; ++e) {
      const int r = r0 + e;
      const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
      const bool ok = i < p.M;
      const long long off = (long long)i * p.ldc + j;
      gin[e] = (EPI == BT_EPI_DGELU && ok) ? p.gelu_in[off] : 0.f;
      res[e] = (has_res && ok) ? p.residual[off] : 0.f;
      old[e] = (has_old && ok) ? p.C[off] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < EC; ++e) {
      const int r = r0 + e;
      const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
      if (i >= p.M) continue;
      const long long off = (long long)i * p.ldc + j;
      float v = acc[r];
      if (EPI == BT_EPI_BIAS) {
        v += bj;
      } else if (EPI == BT_EPI_BIAS_GELU) {
        const float pre = v + bj;
        if (p.preact) p.preact[off] = pre;
        v = gelu_f(pre);
      } else if (EPI == BT_EPI_DGELU) {
        v *= gelu_grad_f(gin[e]);
      }
      v += res[e] + old[e];
      p.C[off] = v;
    }
  }
}

// GELU-backward inputs (pre-activations, with the output's leading
// dimension) of accumulator block b of a wave tile: 16 per lane, in
// accumulator register order, 0 outside the matrix.
template <int NB>
__device__ __forceinline__ void load_gin_block(const GemmParams& p, int b, int im, int jn, int lr, int hh,
                                               float (&g)[16]) {
  const int j = jn + (b % NB) * 32 + lr;
  const int i0 = im + (b / NB) * 32;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
    g[r] = (j < p.N && i < p.M) ? p.gelu_in[(long long)i * p.ldc + j] : 0.f;
  }
}

// Epilogue of a whole wave tile with neither a residual nor an old C to add
// (plain, bias and GELU-backward products).  The only loads are the
// GELU-backward inputs, read a 32 x 32 block at a time one block ahead of
// the stores: loads and stores retire in order on one counter, so waiting
// for inputs issued after a block's stores would also wait for those stores
// to be written (the general path's 4-row groups do exactly that).
template <int EPI, int MB, int NB>
__device__ __forceinline__ void epilogue_plain(const GemmParams& p, const floatx16 (&acc)[MB][NB], int im, int jn,
                                               int lr, int hh, const float (&bj)[NB]) {
  constexpr int NBLK = MB * NB;
  float gin[2][16];
  if (EPI == BT_EPI_DGELU) load_gin_block<NB>(p, 0, im, jn, lr, hh, gin[0]);
#pragma unroll
  for (int b = 0; b < NBLK; ++b) {
    if (EPI == BT_EPI_DGELU && b + 1 < NBLK) load_gin_block<NB>(p, b + 1, im, jn, lr, hh, gin[(b + 1) & 1]);
    const int mb = b / NB, nb = b % NB;
    const int j = jn + nb * 32 + lr;
    if (j >= p.N) continue;
    const int i0 = im + mb * 32;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
      if (i >= p.M) continue;
      float v = acc[mb][nb][r];
      if (EPI == BT_EPI_BIAS) v += bj[nb];
      if (EPI == BT_EPI_DGELU) v *= gelu_grad_f(gin[b & 1][r]);
      p.C[(long long)i * p.ldc + j] = v;
    }
  }
}

// Epilogue of a whole wave tile of a bias product with at most one tensor to
// add, `src` (a residual, or C itself when beta = 1; null: none), streamed
// like the GELU-backward inputs above (every element of C is read before it
// is written).
template <int MB, int NB>
__device__ __forceinline__ void epilogue_bias_add(const GemmParams& p, const float* src,
                                                  const floatx16 (&acc)[MB][NB], int im, int jn, int lr, int hh,
                                                  const float (&bj)[NB]) {
  constexpr int NBLK = MB * NB;
  const bool has_in = src != nullptr;
  float in[2][16];
  auto load = [&](int b, float(&g)[16]) {
    const int j = jn + (b % NB) * 32 + lr;
    const int i0 = im + (b / NB) * 32;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
      g[r] = (j < p.N && i < p.M) ? src[(long long)i * p.ldc + j] : 0.f;
    }
  };
  if (has_in) load(0, in[0]);
#pragma unroll
  for (int b = 0; b < NBLK; ++b) {
    if (has_in && b + 1 < NBLK) load(b + 1, in[(b + 1) & 1]);
    const int mb = b / NB, nb = b % NB;
    const int j = jn + nb * 32 + lr;
    if (j >= p.N) continue;
    const int i0 = im + mb * 32;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
      if (i >= p.M) continue;
      float v = acc[mb][nb][r] + bj[nb];
      if (has_in) v += in[b & 1][r];
      p.C[(long long)i * p.ldc + j] = v;
    }
  }
}

// WM x WN waves, each owning a (32 MB) x (32 NB) output sub-tile of MB x NB
// MFMA accumulators: block tile (32 MB WM) x (32 NB WN), 64 WM WN threads.  DTL: every tile of the launch is
// full (M, N multiples of the block tile, K range a multiple of BK), and
// operand tiles are copied straight from global memory into LDS; otherwise
// they are staged through registers with bounds checks (ragged shapes).
// BMODE 1 (causal): a batch of products (blockIdx.x % nbatch selects the
// batch) in which the output rows of a tile starting at m0 only sum
// k < m0 + BM; tile rows are launched heaviest first.  BMODE 2 (segmented):
// the same with positions (GemmParams::seg): a row tile sums, in each key
// segment, the prefix of k whose positions do not exceed its last row's, in
// BM-aligned steps.  OCC is the number of waves per SIMD the
// register allocation must allow (the second launch-bounds argument on
// AMDGPU); a CU then holds 4 OCC / (WM WN) blocks.
template <bool A_KC, bool B_KC, int EPI, bool SPLIT, bool COLSUM, int BK, int OCC, int WM, int WN, int MB, int NB,
          bool DTL, int BMODE>
__global__ void __launch_bounds__(64 * WM * WN, OCC) gemm_f32_mfma(const GemmParams pk) {
  GemmParams p = pk;
  constexpr int WTM = 32 * MB, WTN = 32 * NB;  // wave tile: MB x NB MFMA 32x32 blocks
  constexpr int BM = WTM * WM, BN = WTN * WN, NW = WM * WN, NT = 64 * NW;
  constexpr int A_SZ = TileSize<A_KC, BM, BK, DTL>::value;
  constexpr int B_SZ = TileSize<B_KC, BN, BK, DTL>::value;
  constexpr int NVA = DTL ? 1 : TileVecs<BM, BK, NT>::value;  // float4 staged per thread, A
  constexpr int NVB = DTL ? 1 : TileVecs<BN, BK, NT>::value;  // float4 staged per thread, B
  constexpr int CA = BM * BK / (256 * NW);  // direct 1 KB copies per wave per tile, A
  constexpr int CB = BN * BK / (256 * NW);  // direct 1 KB copies per wave per tile, B
  static_assert(!DTL || (CA >= 1 && CB >= 1 && CA * 256 * NW == BM * BK && CB * 256 * NW == BN * BK),
                "direct copies must tile the operand tiles in 1 KB slices");
  static_assert(!DTL || (BM <= 256 && BN <= 256), "an MN-contiguous k-row must fit one wave copy");
  static_assert(DTL || !COLSUM || 4 * NT <= 2 * (A_SZ + B_SZ), "column-sum combine needs 16 B per thread of LDS");
  static_assert(2 * (A_SZ + B_SZ) * 4 * (4 * OCC / NW) <= 160 * 1024, "LDS exceeds one CU at this occupancy");
  __shared__ __attribute__((aligned(16))) float smem[2 * (A_SZ + B_SZ)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lr = lane & 31;
  const int hh = lane >> 5;
  const int wm = wave / WN, wn = wave % WN;

  int z, tm, tn;
  if (BMODE != 0) {
    const int y = blockIdx.x % p.nbatch;
    const int rank = blockIdx.x / p.nbatch;  // 0: last tile row (longest k range)
    tm = p.tiles_m - 1 - rank / p.tiles_n;
    tn = rank % p.tiles_n;
    z = 0;
    const int yb = y / p.batch_h, yh = y % p.batch_h;
    p.A += yb * p.sa_b + yh * p.sa_h;
    p.B += yb * p.sb_b + yh * p.sb_h;
    p.C += yb * p.sc_b + yh * p.sc_h;
  } else {
    // ---- tile scheduling: XCD-contiguous ranges of a grouped tile order
    const int ntiles = p.tiles_m * p.tiles_n;
    const int total = gridDim.x;
    int bid = blockIdx.x;
    if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
    z = bid / ntiles;
    const int tile = bid - z * ntiles;
    const int group = 8 * p.tiles_n;
    const int gid = tile / group;
    const int first_m = gid * 8;
    const int gsz = min(p.tiles_m - first_m, 8);
    const int in_g = tile - gid * group;
    tm = first_m + in_g % gsz;
    tn = in_g / gsz;
  }
  const int m0 = tm * BM, n0 = tn * BN;

  const int kbeg = z * p.ksplit;
  int kend = min(p.K, kbeg + p.ksplit);
  if (BMODE == 1) kend = min(kend, m0 + BM);
  int nk, n0t = 0;  // k-tiles; segmented: k-tiles in the first key segment
  if (BMODE == 2) {
    const int last = (m0 < p.seg ? p.q_pos[0] + m0 : p.q_pos[1] + (m0 - p.seg)) + BM - 1;
    auto visible = [&](int kpos) { return last < kpos ? 0 : min(p.seg, (last - kpos) / BM * BM + BM); };
    n0t = visible(p.k_pos[0]) / BK;
    nk = n0t + (p.K > p.seg ? visible(p.k_pos[1]) / BK : 0);
  } else {
    nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  }
  // k offset (from kbeg) of k-tile t
  auto koff = [&](int t) { return BMODE == 2 ? (t < n0t ? t * BK : p.seg + (t - n0t) * BK) : t * BK; };

  // bias of this lane's output columns, loaded before the k-loop so that
  // the epilogue never waits for it behind its own stores
  float bias_j[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int j = n0 + wn * WTN + nb * 32 + lr;
    bias_j[nb] = ((EPI == BT_EPI_BIAS || EPI == BT_EPI_BIAS_GELU) && !SPLIT && j < p.N) ? p.bias[j] : 0.f;
  }
  floatx16 acc[MB][NB];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  floatx4 ra[NVA], rb[NVB];
  unsigned oa[CA], ob[CB];
  const long long a_unit = A_KC ? 1 : p.lda;  // source advance per unit of k
  const long long b_unit = B_KC ? 1 : p.ldb;
  // Column sums of op(B) (only for MN-contiguous B, i.e. op(B) = B [K][N]),
  // kept only by the first tile row of blocks (tm == 0).  Staged path: each
  // thread adds up the B rows it stages and the NT / (BN/4) row groups are
  // combined at the end.  Direct path: each lane adds up the B fragments it
  // reads (its column, its half of every k-tile) and the lane halves are
  // combined at the end.
  floatx4 csum = floatx4{0.f, 0.f, 0.f, 0.f};
  floatx4 csf[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) csf[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  // direct copies: per-lane offsets, the block's operand bases at kbeg and
  // the LDS byte addresses of this wave's slices, all but the offsets scalar
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const float* const a_blk = p.A + (A_KC ? (long long)m0 * p.lda + kbeg : (long long)kbeg * p.lda + m0);
  const float* const b_blk = p.B + (B_KC ? (long long)n0 * p.ldb + kbeg : (long long)kbeg * p.ldb + n0);
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) float*)smem;
  const unsigned lds_a = lds0 + 1024u * CA * wave_u, lds_b = lds0 + 4u * A_SZ + 1024u * CB * wave_u;
  constexpr unsigned BUF_BYTES = 4u * (A_SZ + B_SZ);
  if (DTL) {
    copy_offsets<A_KC, BM, BK, CA>(oa, p.lda, wave_u, lane);
    copy_offsets<B_KC, BN, BK, CB>(ob, p.ldb, wave_u, lane);
  }
  if (nk > 0) {
    if (DTL) {
      copy_issue<CA>(a_blk + koff(0) * a_unit, oa, lds_a);
      copy_issue<CB>(b_blk + koff(0) * b_unit, ob, lds_b);
      wait_copies();
    } else {
      load_tile<A_KC, BM, BK, NT>(ra, p.A, p.lda, m0, p.M, kbeg + koff(0), kend, tid);
      load_tile<B_KC, BN, BK, NT>(rb, p.B, p.ldb, n0, p.N, kbeg + koff(0), kend, tid);
      if (COLSUM && tm == 0)
#pragma unroll
        for (int i = 0; i < NVB; ++i) csum += rb[i];
      store_tile<A_KC, BM, BK, NT>(smem, ra, tid);
      store_tile<B_KC, BN, BK, NT>(smem + A_SZ, rb, tid);
    }
  }
  __syncthreads();

  // Column sums are kept by the first tile row of blocks only (tm == 0), and
  // in the direct-copy path by its first wave row (the waves that combine
  // them at the end); everyone else skips the adds (a uniform branch).
  const bool cs_block = COLSUM && tm == 0;
  const bool cs_wave = cs_block && wm == 0;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      if (DTL) {
        // the other buffer was last read before the previous barrier
        copy_issue<CA>(a_blk + koff(kt + 1) * a_unit, oa, lds_a + (cur ^ 1) * BUF_BYTES);
        copy_issue<CB>(b_blk + koff(kt + 1) * b_unit, ob, lds_b + (cur ^ 1) * BUF_BYTES);
      } else {
        const int k0 = kbeg + koff(kt + 1);
        load_tile<A_KC, BM, BK, NT>(ra, p.A, p.lda, m0, p.M, k0, kend, tid);
        load_tile<B_KC, BN, BK, NT>(rb, p.B, p.ldb, n0, p.N, k0, kend, tid);
      }
    }
    const float* sA = smem + cur * (A_SZ + B_SZ);
    const float* sB = sA + A_SZ;
    // raised wave priority while this wave issues its MFMAs, so the
    // arbiter favours waves that keep the matrix core fed over waves that
    // are staging the next tile
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int c = 0; c < BK / 8; ++c) {
      const int koff = 8 * hh + 4 * (c & 1) + 16 * (c >> 1);
      floatx4 fa[MB], fb[NB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) fa[mb] = read_frag<A_KC, BM, BK, DTL>(sA, wm * WTM + mb * 32 + lr, koff);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fb[nb] = read_frag<B_KC, BN, BK, DTL>(sB, wn * WTN + nb * 32 + lr, koff);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[mb][q], fb[nb][q], acc[mb][nb],
                                                               0, 0, 0);
      if (DTL && COLSUM && cs_wave) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) csf[nb] += fb[nb];
      }
    }
    __builtin_amdgcn_s_setprio(0);
    if (DTL) {
      wait_copies();
    } else if (more) {
      if (COLSUM && cs_block)
#pragma unroll
        for (int i = 0; i < NVB; ++i) csum += rb[i];
      float* sN = smem + (cur ^ 1) * (A_SZ + B_SZ);
      store_tile<A_KC, BM, BK, NT>(sN, ra, tid);
      store_tile<B_KC, BN, BK, NT>(sN + A_SZ, rb, tid);
    }
    __syncthreads();
  }

  if (COLSUM && tm == 0) {
    if (DTL) {
      // waves of the first wave row read every B column of the tile once
      if (wm == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          float v = (csf[nb][0] + csf[nb][1]) + (csf[nb][2] + csf[nb][3]);
          v += __shfl_xor(v, 32, 64);
          const int n = n0 + wn * WTN + nb * 32 + lr;
          if (hh == 0 && n < p.N) {
            if (SPLIT) {
              p.ws_colsum[(long long)z * p.N + n] = v;
            } else {
              if (p.beta != 0.f) v += p.colsum[n];
              p.colsum[n] = v;
            }
          }
        }
      }
    } else {
      // combine the staging row groups (tid / (BN/4)) in a fixed order
      constexpr int TPK = BN / 4, GROUPS = NT / TPK;
      floatx4* red = reinterpret_cast<floatx4*>(smem);
      red[tid] = csum;
      __syncthreads();
      if (tid < TPK) {
        floatx4 s = red[tid];
#pragma unroll
        for (int gi = 1; gi < GROUPS; ++gi) s += red[tid + TPK * gi];
        const int n = n0 + 4 * tid;
        if (n < p.N) {
          if (SPLIT) {
            *reinterpret_cast<floatx4*>(p.ws_colsum + (long long)z * p.N + n) = s;
          } else {
            floatx4* d = reinterpret_cast<floatx4*>(p.colsum + n);
            if (p.beta != 0.f) s += *d;
            *d = s;
          }
        }
      }
    }
  }

  // ---- epilogue.  Accumulator element r of lane (lr, hh) of block (mb, nb):
  // row = 8 (r/4) + 4 hh + r%4, column = lr.
  // Streamed epilogues: plain and GELU-backward products without additive
  // inputs, and bias products with at most one additive input (residual or
  // beta = 1, chosen at run time).  The rest (two additive inputs, additive
  // inputs on the other epilogues, and the bias + GELU products, which also
  // store the pre-activation) take the general path: streaming there spills
  // at 4 waves per SIMD, and a run-time input on the plain products measured
  // 1-4% slower.
  if constexpr (!SPLIT && EPI == BT_EPI_BIAS) {
    if (p.residual == nullptr || p.beta == 0.f) {
      const float* src = p.residual ? p.residual : (p.beta != 0.f ? p.C : nullptr);
      epilogue_bias_add<MB, NB>(p, src, acc, m0 + wm * WTM, n0 + wn * WTN, lr, hh, bias_j);
      return;
    }
  }
  if (!SPLIT && EPI != BT_EPI_BIAS && EPI != BT_EPI_BIAS_GELU && p.residual == nullptr && p.beta == 0.f) {
    epilogue_plain<EPI, MB, NB>(p, acc, m0 + wm * WTM, n0 + wn * WTN, lr, hh, bias_j);
    return;
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int j = n0 + wn * WTN + nb * 32 + lr;
      const int i0 = m0 + wm * WTM + mb * 32;
      if (SPLIT) {
        if (j >= p.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = i0 + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (i < p.M) p.ws[(long long)z * p.M * p.N + (long long)i * p.N + j] = acc[mb][nb][r];
        }
      } else {
        epilogue_block<EPI>(p, acc[mb][nb], i0, j, hh, bias_j[nb]);
      }
    }
}

// Fixed-order sum of split-K partials, then the product's epilogue, element
// by element in the tile epilogue's order: v = sum_z ws[z]; bias (+ GELU,
// storing the pre-activation) or the GELU-backward factor; + residual +
// beta * C.
template <int EPI>
__global__ void __launch_bounds__(256) splitk_reduce(const GemmParams p) {
  const float* __restrict__ ws = p.ws;
  const int M = p.M, N = p.N, splits = p.splits;
  const long long n4 = (long long)M * (N / 4);
  const long long MN = (long long)M * N;
  // column sums of op(B) (bias gradient): colsum = sum_z ws_colsum[z] +
  // beta colsum, in the same fixed order
  if (p.colsum != nullptr) {
    for (int n = blockIdx.x * blockDim.x + threadIdx.x; n < N; n += gridDim.x * blockDim.x) {
      float s = p.ws_colsum[n];
      for (int z = 1; z < splits; ++z) s += p.ws_colsum[(long long)z * N + n];
      if (p.beta != 0.f) s += p.colsum[n];
      p.colsum[n] = s;
    }
  }
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < n4;
       e += (long long)gridDim.x * blockDim.x) {
    const int i = (int)(e / (N / 4));
    const int j = (int)(e - (long long)i * (N / 4)) * 4;
    const float* w = ws + (long long)i * N + j;
    floatx4 v = *reinterpret_cast<const floatx4*>(w);
    for (int z = 1; z < splits; ++z) v += *reinterpret_cast<const floatx4*>(w + z * MN);
    const long long off = (long long)i * p.ldc + j;
    // bias, pre-activation, GELU input and residual carry no alignment
    // requirement beyond 4 bytes: element accesses
    if (EPI == BT_EPI_BIAS || EPI == BT_EPI_BIAS_GELU) {
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] += p.bias[j + k];
      if (EPI == BT_EPI_BIAS_GELU) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (p.preact) p.preact[off + k] = v[k];
          v[k] = gelu_f(v[k]);
        }
      }
    } else if (EPI == BT_EPI_DGELU) {
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] *= gelu_grad_f(p.gelu_in[off + k]);
    }
    floatx4* c = reinterpret_cast<floatx4*>(p.C + off);
    floatx4 add = floatx4{0.f, 0.f, 0.f, 0.f};
    if (p.residual) {
#pragma unroll
      for (int k = 0; k < 4; ++k) add[k] = p.residual[off + k];
    }
    if (p.beta != 0.f) add += *c;
    *c = v + add;
  }
}


// Block-tile configurations: tile depth, wave grid (64 x 64 outputs per
// wave), 32 x 32 blocks per wave, resident blocks per CU (= waves per SIMD
// for 4-wave blocks), and the launch model's constants, fitted on MI355X to
// the measured time of every (tile, split) choice of the products of three
// GPT-2 training steps (124M at 16384 tokens, 124M at 32768, 2.42B at 2048;
// 1100 timings, 3.8% rms error; a fit without any one of the three picks
// within 0.5% of the best measured choice on it):
//  rate_kc / rate_mn  relative k-loop rate with a K-contiguous operand /
//                     with both operands MN-contiguous;
//  ovh                a block's cost outside the k-loop (pipeline fill,
//                     epilogue, and the partial tile's round trip through
//                     the workspace when split), in 128 x 128 x 16 steps;
//  part[q]            rate of a last round in which a CU holds (q+1)/4 of
//                     its full complement of blocks.
// Larger block tiles (256 x 128, 128 x 256, 256 x 256 with 64 x 64 per
// wave) and larger wave tiles (64 x 128 or 128 x 64 at 2 waves per SIMD;
// 128 x 128 spills) were measured slower on most of the model's shapes and
// are not offered.
struct TileCfg {
  int bk, wm, wn, mb, nb, occ;
  double rate_kc, rate_mn, ovh;
  double part[3];
};
constexpr TileCfg kTileCfgs[] = {
    {32, 2, 2, 2, 2, 2, 1.031, 1.013, 6.11, {0.90, 0.90, 0.90}},
    {16, 2, 2, 2, 2, 4, 1.046, 1.038, 5.76, {0.88, 0.974, 0.987}},
};
constexpr int NUM_TILE_CFGS = (int)(sizeof(kTileCfgs) / sizeof(kTileCfgs[0]));

struct GemmCfg {
  int tc;  // index into kTileCfgs
  int splits, ksplit;
};

// Relative time of a launch of `blocks` equal blocks (each `work` long) on
// tile configuration c: the busiest CU holds ceil(blocks / NUM_CU) of them
// and runs up to `occ` at once; a last, partial round runs at c.part[].
double launch_time(const TileCfg& c, long long blocks, double work) {
  const int occ = c.occ * 4 / (c.wm * c.wn);
  const long long per_cu = (blocks + NUM_CU - 1) / NUM_CU;
  const long long full = per_cu / occ, rem = per_cu % occ;
  double t = (double)(full * occ) * work;
  if (rem) {
    int q = (int)((4 * rem + occ / 2) / occ) - 1;
    q = q < 0 ? 0 : q > 2 ? 2 : q;
    t += (double)rem * work / c.part[q];
  }
  return t;
}

// Tile configuration and K split for a shape (a split product's epilogue
// runs in the reduction of the partials).
GemmCfg choose_config(int M, int N, int K, bool akc, bool bkc, bool may_split) {
  if (K <= 0) return GemmCfg{0, 1, 32};
  // Very long k-loops over K-contiguous rows of A with at least two tiles
  // per CU (the LM head's input gradient: K = 50304, 768 tiles) run faster
  // on the deeper tile, split as the model chooses: measured on MI355X at
  // 86-87% of the matrix peak vs 81-84% on the 16-deep tile.
  const bool deep_only = K >= 32768 && akc && (long long)((M + 127) / 128) * ((N + 127) / 128) >= 2 * NUM_CU;
  GemmCfg best{0, 1, K};
  double best_t = 1e300;
  // a near tie (within 0.5%) keeps the configuration met first: the one
  // with more resident blocks, then the smaller split
  for (int tc = NUM_TILE_CFGS - 1; tc >= 0; --tc) {
    if (deep_only && kTileCfgs[tc].bk != 32) continue;
    // with both operands MN-contiguous the 32-deep tile is slower at every
    // block count (its rate_mn and per-block cost are both worse); it is not
    // built for that layout
    if (!akc && !bkc && kTileCfgs[tc].bk != 16) continue;
    const TileCfg& c = kTileCfgs[tc];
    const int bm = 32 * c.mb * c.wm, bn = 32 * c.nb * c.wn, bk = c.bk;
    const long long tiles = (long long)((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    const int kt = (K + bk - 1) / bk;
    int smax = 1;
    if (may_split && K >= 8 * bk) smax = kt / 4 < 32 ? kt / 4 : 32;
    for (int s = 1; s <= smax; ++s) {
      int ks = (K + s - 1) / s;
      ks = (ks + bk - 1) / bk * bk;
      if ((K + ks - 1) / ks != s) continue;
      if (s > 1 && (double)s * M * N * sizeof(float) > (double)MAX_SPLIT_WS) continue;
      // time in 128 x 128 x 16 tile steps of a full CU
      const double work =
          (double)bm * bn / (128.0 * 128.0) * (ks / 16.0 / ((akc || bkc) ? c.rate_kc : c.rate_mn) + c.ovh);
      const double t = launch_time(c, tiles * s, work);
      if (t < best_t * 0.995) {
        best_t = t;
        best = GemmCfg{tc, s, ks};
      }
    }
  }
  return best;
}

template <bool A_KC, bool B_KC, int BK, int OCC, int WM, int WN, int MB, int NB, bool DTL>
void launch_cfg(const GemmParams& p, int epi, bool split, dim3 grid, hipStream_t s) {
  const bool cs = p.colsum != nullptr;
  const dim3 block(64 * WM * WN);
  if (split) {
    if (cs)
      hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_NONE, true, !B_KC, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
    else
      hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_NONE, true, false, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
    return;
  }
  switch (epi) {
    case BT_EPI_NONE:
      if (cs)
        hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_NONE, false, !B_KC, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
      else
        hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_NONE, false, false, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
      break;
    case BT_EPI_BIAS:
      hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_BIAS, false, false, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
      break;
    case BT_EPI_BIAS_GELU:
      hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_BIAS_GELU, false, false, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
      break;
    default:
      hipLaunchKernelGGL((gemm_f32_mfma<A_KC, B_KC, BT_EPI_DGELU, false, false, BK, OCC, WM, WN, MB, NB, DTL, 0>), grid, block, 0, s, p);
      break;
  }
}

// dtl: every tile is full, so operand tiles are copied directly into LDS
template <bool A_KC, bool B_KC>
void launch_layout(const GemmParams& p, const GemmCfg& c, int epi, bool split, bool dtl, dim3 grid,
                   hipStream_t s) {
#define BT_GEMM_CFG(BK_, OCC_, WM_, WN_, MB_, NB_)                                         \
  if (dtl) launch_cfg<A_KC, B_KC, BK_, OCC_, WM_, WN_, MB_, NB_, true>(p, epi, split, grid, s); \
  else launch_cfg<A_KC, B_KC, BK_, OCC_, WM_, WN_, MB_, NB_, false>(p, epi, split, grid, s)
  if constexpr (A_KC || B_KC) {
    if (c.tc == 0) {
      BT_GEMM_CFG(32, 2, 2, 2, 2, 2);
      return;
    }
  }
  BT_GEMM_CFG(16, 4, 2, 2, 2, 2);
#undef BT_GEMM_CFG
}

}  // namespace

// One configuration of the batched causal / segmented product: a
// (32 MB WM) x (32 NB WN) block tile of WM x WN waves, each wave a
// (32 MB) x (32 NB) tile.
template <int BMODE, int WM, int WN, int MB, int NB, int OCC>
static bt_status launch_batched(GemmParams p, hipStream_t stream) {
  constexpr int BK = 16, BM = 32 * MB * WM, BN = 32 * NB * WN;
  p.ksplit = (p.K + BK - 1) / BK * BK;
  p.splits = 1;
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const long long nblocks = (long long)p.tiles_m * p.tiles_n * p.nbatch;
  BT_RETURN_IF(nblocks > 0x7fffffffLL, BT_ESHAPE, "batched product: too many tiles");
  const bool dtl = p.M % BM == 0 && p.N % BN == 0 && p.K % BK == 0 && copy_offsets_fit(p.lda, p.ldb);
  if (dtl)
    hipLaunchKernelGGL((gemm_f32_mfma<true, false, BT_EPI_NONE, false, false, BK, OCC, WM, WN, MB, NB, true, BMODE>),
                       dim3((unsigned)nblocks), dim3(64 * WM * WN), 0, stream, p);
  else
    hipLaunchKernelGGL((gemm_f32_mfma<true, false, BT_EPI_NONE, false, false, BK, OCC, WM, WN, MB, NB, false, BMODE>),
                       dim3((unsigned)nblocks), dim3(64 * WM * WN), 0, stream, p);
  return check_launch(BMODE == 1 ? "gemm_f32_mfma (batched causal)" : "gemm_f32_mfma (batched segmented)");
}

static bt_status batched_params(GemmParams* p, const char* who, int M, int N, int K, const float* A, int lda,
                                long long sa_b, long long sa_h, const float* B, int ldb, long long sb_b,
                                long long sb_h, float* C, int ldc, long long sc_b, long long sc_h, int nb,
                                int nh) {
  BT_RETURN_IF(M <= 0 || N <= 0 || K <= 0 || nb <= 0 || nh <= 0, BT_ESHAPE,
               "%s: bad sizes M=%d N=%d K=%d nb=%d nh=%d", who, M, N, K, nb, nh);
  BT_RETURN_IF((M | N | K | lda | ldb | ldc) & 3, BT_ESHAPE, "%s: sizes and strides must be multiples of 4", who);
  BT_RETURN_IF(!aligned16(A) || !aligned16(B) || !aligned16(C) || ((sa_b | sa_h | sb_b | sb_h | sc_b | sc_h) & 3),
               BT_EALIGN, "%s: operands must be 16-byte aligned", who);
  *p = GemmParams{};
  p->A = A;
  p->B = B;
  p->C = C;
  p->lda = lda;
  p->ldb = ldb;
  p->ldc = ldc;
  p->M = M;
  p->N = N;
  p->K = K;
  p->nbatch = nb * nh;
  p->batch_h = nh;
  p->sa_b = sa_b;
  p->sa_h = sa_h;
  p->sb_b = sb_b;
  p->sb_h = sb_h;
  p->sc_b = sc_b;
  p->sc_h = sc_h;
  return BT_OK;
}

bt_status gemm_causal_batched(int M, int N, int K, const float* A, int lda, long long sa_b, long long sa_h,
                              const float* B, int ldb, long long sb_b, long long sb_h, float* C, int ldc,
                              long long sc_b, long long sc_h, int nb, int nh, hipStream_t stream) {
  GemmParams p;
  BT_TRY(batched_params(&p, "gemm_causal_batched", M, N, K, A, lda, sa_b, sa_h, B, ldb, sb_b, sb_h, C, ldc, sc_b,
                        sc_h, nb, nh));
  // Both use 128 x 64 block tiles.  Up to T = 8192 rows, four waves of 64 x 32
  // (one wave per SIMD guaranteed, so the register budget is the full file)
  // hide latency better: measured 8-14% faster on MI355X at T = 1024 and
  // 4096.  At T = 16384 each tile's K loop is long enough that two waves of
  // 64 x 64, with their higher arithmetic intensity per LDS read, win by ~1%.
  if (M <= 8192) return launch_batched<1, 2, 2, 2, 1, 1>(p, stream);
  return launch_batched<1, 2, 1, 2, 2, 2>(p, stream);
}

bt_status gemm_segmented_batched(int M, int N, int K, const float* A, int lda, long long sa_b, long long sa_h,
                                 const float* B, int ldb, long long sb_b, long long sb_h, float* C, int ldc,
                                 long long sc_b, long long sc_h, int nb, int nh, float beta, int seg,
                                 const int* q_pos, const int* k_pos, hipStream_t stream) {
  GemmParams p;
  BT_TRY(batched_params(&p, "gemm_segmented_batched", M, N, K, A, lda, sa_b, sa_h, B, ldb, sb_b, sb_h, C, ldc,
                        sc_b, sc_h, nb, nh));
  constexpr int BM = 128;  // row tile of both configurations below
  BT_RETURN_IF(seg <= 0 || seg % BM || M % seg || K % seg || M / seg > 2 || K / seg > 2, BT_ESHAPE,
               "gemm_segmented_batched: segments of %d rows must be multiples of %d and 1 or 2 per side", seg, BM);
  for (int i = 0; i < 2; ++i) {
    BT_RETURN_IF(i < M / seg && (q_pos[i] < 0 || q_pos[i] % BM), BT_ESHAPE, "gemm_segmented_batched: bad position");
    BT_RETURN_IF(i < K / seg && (k_pos[i] < 0 || k_pos[i] % BM), BT_ESHAPE, "gemm_segmented_batched: bad position");
    p.q_pos[i] = i < M / seg ? q_pos[i] : 0;
    p.k_pos[i] = i < K / seg ? k_pos[i] : 0;
  }
  BT_RETURN_IF(beta != 0.f && beta != 1.f, BT_EINVAL, "gemm_segmented_batched: beta must be 0 or 1");
  p.seg = seg;
  p.beta = beta;
  if (M <= 8192) return launch_batched<2, 2, 2, 2, 1, 1>(p, stream);
  return launch_batched<2, 2, 1, 2, 2, 2>(p, stream);
}

}  // namespace bt

using namespace bt;

namespace bt {
namespace {
// Direct global-to-LDS operand copies: every tile of the launch is full and
// the per-lane copy offsets fit their 32-bit registers.
bool direct_tiles(const GemmCfg& cfg, int M, int N, int K, int lda, int ldb) {
  const TileCfg& t = kTileCfgs[cfg.tc];
  return M % (32 * t.mb * t.wm) == 0 && N % (32 * t.nb * t.wn) == 0 && K % t.bk == 0 && copy_offsets_fit(lda, ldb);
}
}  // namespace
}  // namespace bt

extern "C" bt_status bt_gemm_plan(bt_op opA, bt_op opB, int M, int N, int K, int lda, int ldb, int* tile_depth,
                                  int* splits, int* direct) {
  bt::clear_error();
  BT_RETURN_IF(opA != BT_OP_N && opA != BT_OP_T, BT_EINVAL, "bt_gemm_plan: bad opA %d", (int)opA);
  BT_RETURN_IF(opB != BT_OP_N && opB != BT_OP_T, BT_EINVAL, "bt_gemm_plan: bad opB %d", (int)opB);
  BT_RETURN_IF(M <= 0 || N <= 0 || K <= 0 || ((M | N | K) & 3), BT_ESHAPE,
               "bt_gemm_plan: M=%d N=%d K=%d must be positive multiples of 4", M, N, K);
  BT_RETURN_IF(!tile_depth || !splits || !direct, BT_EINVAL, "bt_gemm_plan: NULL output");
  const GemmCfg c = choose_config(M, N, K, opA == BT_OP_N, opB == BT_OP_T, true);
  *tile_depth = kTileCfgs[c.tc].bk;
  *splits = c.splits;
  *direct = direct_tiles(c, M, N, K, lda, ldb) ? 1 : 0;
  return BT_OK;
}

extern "C" size_t bt_gemm_ws_bytes(bt_op opA, bt_op opB, int M, int N, int K, bt_epi epi) {
  if (M <= 0 || N <= 0 || K <= 0 || epi < BT_EPI_NONE || epi > BT_EPI_DGELU) return 0;
  const GemmCfg c = choose_config(M, N, K, opA == BT_OP_N, opB == BT_OP_T, true);
  const int splits = c.splits;
  if (splits <= 1) return 0;
  return (size_t)splits * ((size_t)M * N + N) * sizeof(float);
}

extern "C" bt_status bt_gemm(bt_op opA, bt_op opB, int M, int N, int K, const float* A, int lda,
                             const float* B, int ldb, float beta, float* C, int ldc,
                             const float* bias, bt_epi epi, float* preact_out,
                             const float* gelu_in, const float* residual, float* colsum_B, void* ws,
                             size_t ws_bytes, void* stream) {
  bt::clear_error();
  BT_RETURN_IF(opA != BT_OP_N && opA != BT_OP_T, BT_EINVAL, "bt_gemm: bad opA %d", (int)opA);
  BT_RETURN_IF(opB != BT_OP_N && opB != BT_OP_T, BT_EINVAL, "bt_gemm: bad opB %d", (int)opB);
  BT_RETURN_IF(epi < BT_EPI_NONE || epi > BT_EPI_DGELU, BT_EINVAL, "bt_gemm: bad epilogue %d", (int)epi);
  BT_RETURN_IF(M < 0 || N < 0 || K < 0, BT_ESHAPE, "bt_gemm: negative size M=%d N=%d K=%d", M, N, K);
  BT_RETURN_IF((M | N | K) & 3, BT_ESHAPE, "bt_gemm: M=%d N=%d K=%d must be multiples of 4", M, N, K);
  BT_RETURN_IF(beta != 0.f && beta != 1.f, BT_EINVAL, "bt_gemm: beta must be 0 or 1 (got %g)", beta);
  if (M == 0 || N == 0) return BT_OK;
  const int a_cols = opA == BT_OP_N ? K : M;
  const int b_cols = opB == BT_OP_N ? N : K;
  BT_RETURN_IF(lda < a_cols || ldb < b_cols || ldc < N, BT_ESHAPE,
               "bt_gemm: leading dimension too small (lda=%d need %d, ldb=%d need %d, ldc=%d need %d)",
               lda, a_cols, ldb, b_cols, ldc, N);
  BT_RETURN_IF((lda | ldb | ldc) & 3, BT_EALIGN, "bt_gemm: lda/ldb/ldc must be multiples of 4");
  BT_RETURN_IF(!C, BT_EINVAL, "bt_gemm: C is NULL");
  BT_RETURN_IF(K > 0 && (!A || !B), BT_EINVAL, "bt_gemm: A or B is NULL");
  BT_RETURN_IF(!aligned16(C) || (A && !aligned16(A)) || (B && !aligned16(B)), BT_EALIGN,
               "bt_gemm: A, B, C must be 16-byte aligned");
  BT_RETURN_IF((epi == BT_EPI_BIAS || epi == BT_EPI_BIAS_GELU) && !bias, BT_EINVAL,
               "bt_gemm: bias required for this epilogue");
  BT_RETURN_IF(epi == BT_EPI_DGELU && !gelu_in, BT_EINVAL, "bt_gemm: gelu_in required for DGELU");
  BT_RETURN_IF(residual && residual == C, BT_EINVAL, "bt_gemm: residual must not alias C");
  BT_RETURN_IF(colsum_B && (opB != BT_OP_N || epi != BT_EPI_NONE || residual), BT_EINVAL,
               "bt_gemm: colsum_B needs opB = N, no epilogue and no residual");
  BT_RETURN_IF(colsum_B && !aligned16(colsum_B), BT_EALIGN, "bt_gemm: colsum_B must be 16-byte aligned");

  GemmParams p{};
  p.A = A;
  p.B = B;
  p.C = C;
  p.bias = bias;
  p.preact = epi == BT_EPI_BIAS_GELU ? preact_out : nullptr;
  p.gelu_in = gelu_in;
  p.residual = residual;
  p.colsum = colsum_B;
  p.lda = lda;
  p.ldb = ldb;
  p.ldc = ldc;
  p.M = M;
  p.N = N;
  p.K = K;
  p.beta = beta;
  const bool akc = opA == BT_OP_N;
  const bool bkc = opB == BT_OP_T;
  const GemmCfg cfg = choose_config(M, N, K, akc, bkc, true);
  const TileCfg& tcf = kTileCfgs[cfg.tc];
  const int bm = 32 * tcf.mb * tcf.wm, bn = 32 * tcf.nb * tcf.wn;
  p.tiles_m = (M + bm - 1) / bm;
  p.tiles_n = (N + bn - 1) / bn;
  const int splits = cfg.splits;
  p.ksplit = cfg.ksplit;
  p.splits = splits;
  const bool split = splits > 1;
  if (split) {
    const size_t need = (size_t)splits * ((size_t)M * N + N) * sizeof(float);
    BT_RETURN_IF(!ws || ws_bytes < need, BT_EWORKSPACE,
                 "bt_gemm: workspace of %zu bytes needed (got %zu)", need, ws_bytes);
    BT_RETURN_IF(!aligned16(ws), BT_EALIGN, "bt_gemm: workspace must be 16-byte aligned");
    p.ws = static_cast<float*>(ws);
    p.ws_colsum = p.ws + (size_t)splits * M * N;
  }
  const long long nblocks = (long long)p.tiles_m * p.tiles_n * splits;
  BT_RETURN_IF(nblocks > 0x7fffffffLL, BT_ESHAPE, "bt_gemm: too many tiles");
  dim3 grid((unsigned)nblocks);
  hipStream_t s = as_stream(stream);
  const bool dtl = direct_tiles(cfg, M, N, K, lda, ldb);
  if (akc && !bkc) launch_layout<true, false>(p, cfg, epi, split, dtl, grid, s);
  else if (akc && bkc) launch_layout<true, true>(p, cfg, epi, split, dtl, grid, s);
  else if (!akc && !bkc) launch_layout<false, false>(p, cfg, epi, split, dtl, grid, s);
  else launch_layout<false, true>(p, cfg, epi, split, dtl, grid, s);
  BT_TRY(check_launch("gemm_f32_mfma"));
  if (split) {
    const long long n4 = (long long)M * (N / 4);
    long long nb = (n4 + 255) / 256;
    if (nb > 4096) nb = 4096;
    switch (epi) {
      case BT_EPI_NONE: hipLaunchKernelGGL(splitk_reduce<BT_EPI_NONE>, dim3((unsigned)nb), dim3(256), 0, s, p); break;
      case BT_EPI_BIAS: hipLaunchKernelGGL(splitk_reduce<BT_EPI_BIAS>, dim3((unsigned)nb), dim3(256), 0, s, p); break;
      case BT_EPI_BIAS_GELU:
        hipLaunchKernelGGL(splitk_reduce<BT_EPI_BIAS_GELU>, dim3((unsigned)nb), dim3(256), 0, s, p);
        break;
      default: hipLaunchKernelGGL(splitk_reduce<BT_EPI_DGELU>, dim3((unsigned)nb), dim3(256), 0, s, p); break;
    }
    BT_TRY(check_launch("splitk_reduce"));
  }
  return BT_OK;
}

// ---------------------------------------------------------------------------
// bt_gemm without a caller workspace: the split-K partials live in a static
// device array of this library (each GPU the library runs on holds its own
// copy until the process ends).  In host code `gemm_scratch` names a host-side
// stand-in, not the device memory: the device address is looked up once per
// device with hipGetSymbolAddress and only that address is passed to kernels.
namespace {

constexpr size_t GEMM_SCRATCH_BYTES = 64ull << 20;
__device__ __align__(256) char gemm_scratch[GEMM_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

bt_status scratch_address(void** out) {
  int dev = 0;
  BT_CHECK_HIP(hipGetDevice(&dev));
  BT_RETURN_IF(dev < 0 || dev >= MAX_DEVICES, BT_EINVAL, "bt_gemm_noalloc: device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    BT_CHECK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(gemm_scratch)));
    BT_RETURN_IF(!p, BT_EHIP, "bt_gemm_noalloc: no device address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return BT_OK;
}

}  // namespace

extern "C" size_t bt_gemm_noalloc_max_ws_bytes(void) { return GEMM_SCRATCH_BYTES; }

extern "C" bt_status bt_gemm_noalloc(bt_op opA, bt_op opB, int M, int N, int K, const float* A, int lda,
                                     const float* B, int ldb, float beta, float* C, int ldc, const float* bias,
                                     bt_epi epi, float* preact_out, const float* gelu_in, const float* residual,
                                     float* colsum_B, void* stream) {
  bt::clear_error();
  const size_t need = bt_gemm_ws_bytes(opA, opB, M, N, K, epi);
  BT_RETURN_IF(need > GEMM_SCRATCH_BYTES, BT_EWORKSPACE,
               "bt_gemm_noalloc: M=%d N=%d K=%d needs %zu bytes of split-K scratch; the library's static scratch "
               "holds %zu (use bt_gemm with a workspace)", M, N, K, need, GEMM_SCRATCH_BYTES);
  void* ws = nullptr;
  if (need > 0) BT_TRY(scratch_address(&ws));
  return bt_gemm(opA, opB, M, N, K, A, lda, B, ldb, beta, C, ldc, bias, epi, preact_out, gelu_in, residual,
                 colsum_B, ws, need > 0 ? GEMM_SCRATCH_BYTES : 0, stream);
}
