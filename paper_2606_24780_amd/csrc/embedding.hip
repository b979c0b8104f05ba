// Token + position embeddings with the token table tied to the LM head
// (GPT-2 architecture figure: weight-tied embeddings, learned positions).
//
// Forward: x0[b, t] = wte[tok[b, t]] + wpe[t].
//
// Backward, deterministic (no floating-point atomics):
//   dwte[v] += sum over positions m with tok[m] = v of dx0[m]   (position order)
//   dwpe[t]  = beta dwpe[t] + sum_b dx0[b, t]                  (batch order)
//
// The token index.  The backward needs the positions grouped by token.  One
// 1024-thread workgroup builds that grouping: a stable least-significant-digit
// radix sort of (token, position) on 8-bit digits of the token (two passes
// for a 50,304-row table; inside LDS for up to 16,384 tokens, through global
// memory beyond), each pass ranking 64 entries at a time by wave ballots on
// the digit bits, counting per wave, scanning the 16 x 256 counts and
// scattering in position order.  The sorted list is cut into pieces of P
// entries; for every piece the index also records the pieces where the runs
// (equal tokens) through its first and last entries start and end.  The
// index depends only on the tokens: the training step builds it on a second
// stream while the forward runs.
//
// The backward sum is two launches:
//  * token units (piece p, 64-column slice s; a workgroup takes the slices
//    of one piece so the piece's rows are fetched together): a lane owns one
//    column, loads the piece's P rows of dx0 and the dwte rows of the runs
//    that begin and end inside the piece at once, forms running sums along
//    each run and writes those dwte rows.  A run that crosses piece
//    boundaries leaves one partial per piece it touches (A: the piece's last
//    run continues past it; B: the piece's first run began earlier and ends
//    in it); the Zipf head token (about 14% of the positions) is thereby
//    spread over ~74 pieces x 12 slices instead of one workgroup.
//  * second launch: for every crossing run the unit of its first piece adds
//    the partials in piece order, A[s], ..., A[e-1], B[e], into dwte (the
//    kernel boundary makes the partials of every XCD visible: no fences or
//    flags); position units (2 positions, 256-column slice) load the B rows
//    of a position at once (float4 per lane) and sum them in batch order.
#include "bt_internal.h"

namespace bt {
namespace {

constexpr int SORT_THREADS = 1024;
constexpr int SORT_WAVES = SORT_THREADS / 64;
constexpr int RADIX = 256;
constexpr int PIECE = 32;        // entries of the sorted list per token unit
constexpr int TV = 1;            // floats per lane in token and finish units
constexpr int WPE_T = 2;         // positions per position unit
constexpr int TOK_WAVES = 12;    // column slices (waves) per token-unit workgroup
constexpr int FWD_WAVES = 4;     // rows (one per wave) per gather workgroup

__host__ __device__ int bits_for(long long n) {
  int b = 0;
  while ((1LL << b) < n) ++b;
  return b < 1 ? 1 : b;
}

// ------------------------------------------------------------ index layout
// int32 arrays: skey[M], spos[M] (result), tkey[M], tpos[M] (ping-pong),
// fr_start[np] (start piece of the run holding a piece's first entry),
// lr_start[np], lr_end[np] (start / end piece of the run holding its last
// entry).
struct IndexLayout {
  size_t skey, spos, tkey, tpos, fr_start, lr_start, lr_end, total;
};

IndexLayout index_layout(long long M) {
  const long long np = (M + PIECE - 1) / PIECE;
  IndexLayout L;
  size_t off = 0;
  auto take = [&](long long n) {
    const size_t r = off;
    off += align_up((size_t)n * sizeof(int32_t), 256);
    return r;
  };
  L.skey = take(M);
  L.spos = take(M);
  L.tkey = take(M);
  L.tpos = take(M);
  L.fr_start = take(np);
  L.lr_start = take(np);
  L.lr_end = take(np);
  L.total = off;
  return L;
}

struct IndexPtrs {
  int32_t *skey, *spos, *tkey, *tpos, *fr_start, *lr_start, *lr_end;
};

IndexPtrs index_ptrs(void* base, long long M) {
  const IndexLayout L = index_layout(M);
  char* b = static_cast<char*>(base);
  return IndexPtrs{reinterpret_cast<int32_t*>(b + L.skey),     reinterpret_cast<int32_t*>(b + L.spos),
                   reinterpret_cast<int32_t*>(b + L.tkey),     reinterpret_cast<int32_t*>(b + L.tpos),
                   reinterpret_cast<int32_t*>(b + L.fr_start), reinterpret_cast<int32_t*>(b + L.lr_start),
                   reinterpret_cast<int32_t*>(b + L.lr_end)};
}

// ------------------------------------------------------------------- sort
__device__ __forceinline__ int clamp_tok(int id, int Vp) { return id < 0 ? 0 : (id >= Vp ? Vp - 1 : id); }

// Lanes of the wave (among `valid`) whose digit equals this lane's digit.
// Bit b of the digit selects the lanes whose bit b agrees: ballot_b when set,
// its complement when clear, i.e. ballot_b ^ (bit_b - 1) as a 64-bit mask.
__device__ __forceinline__ unsigned long long match_digit(int d, unsigned long long valid) {
  unsigned long long peers = valid;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const unsigned bit = (d >> b) & 1u;
    const unsigned long long m = __ballot(bit);
    peers &= m ^ ((unsigned long long)bit - 1ull);
  }
  return peers;
}

// Exclusive prefix sum over the 1024 threads of the block.
__device__ __forceinline__ int block_excl_sum(int v, int* lds /*[SORT_WAVES]*/) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(inc, o, 64);
    if (lane >= o) inc += u;
  }
  if (lane == 63) lds[wave] = inc;
  __syncthreads();
  int carry = 0;
  for (int w = 0; w < wave; ++w) carry += lds[w];
  __syncthreads();
  return carry + inc - v;
}

// Inputs of up to LDS_SORT_MAX tokens with ids below 2^16 are sorted inside
// the workgroup's LDS as packed (id << 15 | position) words; longer inputs
// (or larger tables) go through global memory.
constexpr int LDS_SORT_MAX = 16384;

struct SortLds {
  int hist[SORT_WAVES][RADIX];  // digit counts per wave, then running offsets
  int scan[SORT_WAVES];
  unsigned buf[LDS_SORT_MAX];
};

// Per pass a wave holds its entries in registers, SORT_CHUNK per lane (one
// chunk for up to 16,384 tokens; longer inputs loop over chunks and reload).
constexpr int SORT_CHUNK = 16;

__device__ __forceinline__ void sort_load(const int32_t* __restrict__ tok, const int32_t* sk, const int32_t* sp,
                                          int Vp, int cb, int w1, int lane, int (&key)[SORT_CHUNK],
                                          int (&pos)[SORT_CHUNK]) {
#pragma unroll
  for (int q = 0; q < SORT_CHUNK; ++q) {
    const int j = cb + 64 * q + lane;
    key[q] = 0;
    pos[q] = j;
    if (j < w1) {
      if (sk) {
        key[q] = sk[j];
        pos[q] = sp[j];
      } else {
        key[q] = clamp_tok(tok[j], Vp);
      }
    }
  }
}

// Piece boundaries of the sorted list (key_at(i) the token of entry i).  A
// wave owns the same contiguous range as in the sort, a multiple of 64
// entries, so each 64-entry step of a wave holds whole pieces: wave ballots
// give the run starts and ends inside the step, and the last start before it
// / first end after it are carried along the wave and across waves.
template <typename KeyAt>
__device__ void run_info(int M, const IndexPtrs ix, SortLds& sm, KeyAt key_at) {
  static_assert(64 % PIECE == 0, "a wave step holds whole pieces");
  constexpr int NC = 16;  // wave steps held at once
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int R = ((M + SORT_WAVES - 1) / SORT_WAVES + 63) / 64 * 64;
  const int w0 = min(M, wave * R), w1 = min(M, w0 + R);
  // start / end masks of NC steps from cb0 on
  auto masks = [&](int cb0, unsigned long long (&ms)[NC], unsigned long long (&me)[NC]) {
    int k[NC + 2];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int j = cb0 + 64 * c + lane;
      k[c] = j < M ? key_at(j) : -1;  // past w1 too: the neighbour of the wave's last entry
    }
    // the neighbours across step boundaries: entry cb0 - 1 and the entry after each step
    const int jp = cb0 - 1, jn = cb0 + 64 * NC;
    const int kprev = (jp >= 0 && jp < M) ? key_at(jp) : -2;
    const int knext = jn < M ? key_at(jn) : -2;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int j = cb0 + 64 * c + lane;
      const bool ok = j < w1;
      int up = __shfl_up(k[c], 1, 64);
      int dn = __shfl_down(k[c], 1, 64);
      const int prev_last = c > 0 ? __shfl(k[c - 1], 63, 64) : kprev;
      const int next_first = c + 1 < NC ? __shfl(k[c + 1], 0, 64) : knext;
      if (lane == 0) up = prev_last;
      if (lane == 63) dn = next_first;
      if (j + 1 >= M) dn = -2;
      ms[c] = __ballot(ok && k[c] != up);
      me[c] = __ballot(ok && k[c] != dn);
    }
  };
  unsigned long long ms[NC], me[NC];
  int wlast = -1, wfirst = 0x7fffffff;
  for (int cb0 = w0; cb0 < w1; cb0 += 64 * NC) {
    masks(cb0, ms, me);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int cb = cb0 + 64 * c;
      if (ms[c]) wlast = cb + 63 - __builtin_clzll(ms[c]);
      if (me[c] && wfirst == 0x7fffffff) wfirst = cb + __builtin_ctzll(me[c]);
    }
  }
  if (lane == 0) {
    sm.scan[wave] = wlast;
    sm.hist[0][wave] = wfirst;
  }
  __syncthreads();
  int prev = -1, nxt = 0x7fffffff;
  for (int w = 0; w < wave; ++w) prev = max(prev, sm.scan[w]);
  for (int w = SORT_WAVES - 1; w > wave; --w) nxt = min(nxt, sm.hist[0][w]);
  __syncthreads();
  const bool single = w1 - w0 <= 64 * NC;  // the masks of the first sweep are still current
  // last start at or before step offset x (prev when none), first end at or
  // after it (nxt when none)
  auto last_start_le = [&](unsigned long long ms, int cb, int x, int prv) {
    const unsigned long long m = ms & (x >= 63 ? ~0ull : ((2ull << x) - 1ull));
    return m ? cb + 63 - __builtin_clzll(m) : prv;
  };
  for (int cb0 = w0; cb0 < w1; cb0 += 64 * NC) {
    if (!single) masks(cb0, ms, me);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int cb = cb0 + 64 * c;
      if (cb < w1) {
#pragma unroll
        for (int o = 0; o < 64; o += PIECE) {
          if (cb + o < w1) {
            const int jl = min(cb + o + PIECE - 1, w1 - 1);
            if (lane == 0) {
              ix.fr_start[(cb + o) / PIECE] = last_start_le(ms[c], cb, o, prev) / PIECE;
              ix.lr_start[(cb + o) / PIECE] = last_start_le(ms[c], cb, jl - cb, prev) / PIECE;
            }
          }
        }
        prev = last_start_le(ms[c], cb, 63, prev);
      }
    }
  }
  const int nsteps = (w1 - w0 + 63) / 64;
  for (int cb0 = w0 + (nsteps - 1) / NC * NC * 64; cb0 >= w0 && nsteps > 0; cb0 -= 64 * NC) {
    if (!single) masks(cb0, ms, me);
#pragma unroll
    for (int c = NC - 1; c >= 0; --c) {
      const int cb = cb0 + 64 * c;
      if (cb < w1) {
#pragma unroll
        for (int o = 0; o < 64; o += PIECE) {
          if (cb + o < w1) {
            const int jl = min(cb + o + PIECE - 1, w1 - 1);
            const unsigned long long m = me[c] & ~((1ull << (jl - cb)) - 1ull);
            const int le = m ? cb + __builtin_ctzll(m) : nxt;
            if (lane == 0) ix.lr_end[(cb + o) / PIECE] = le / PIECE;
          }
        }
        if (me[c]) nxt = cb + __builtin_ctzll(me[c]);
      }
    }
  }
}

// Exclusive scan of the (digit, wave) counts in sm.hist, digit-major, in place.
__device__ __forceinline__ void scan_hist(SortLds& sm) {
  int v[4], s = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = 4 * threadIdx.x + k;
    v[k] = sm.hist[e & (SORT_WAVES - 1)][e >> 4];
    s += v[k];
  }
  int base = block_excl_sum(s, sm.scan);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = 4 * threadIdx.x + k;
    sm.hist[e & (SORT_WAVES - 1)][e >> 4] = base;
    base += v[k];
  }
  __syncthreads();
}

// Rank of this lane among the lanes of its step with the same digit (low 8
// bits) and the number of such lanes (bits 8-15).
__device__ __forceinline__ unsigned digit_rank(int d, bool ok, unsigned long long lt) {
  const unsigned long long peers = match_digit(d, __ballot(ok));
  return (unsigned)__popcll(peers & lt) | ((unsigned)__popcll(peers) << 8);
}

// Counting step: the last lane of each digit group adds the group's size
// (one LDS add per distinct digit, no conflicting lanes).
__device__ __forceinline__ void count_step(SortLds& sm, int wave, int d, bool ok, unsigned rc) {
  const unsigned rank = rc & 255u, cnt = rc >> 8;
  if (ok && rank == cnt - 1) atomicAdd(&sm.hist[wave][d], (int)cnt);
}

// Scatter step: the group's slots start at the digit's running offset,
// which the group's last lane then advances.
__device__ __forceinline__ int scatter_step(SortLds& sm, int wave, int d, bool ok, unsigned rc) {
  const unsigned rank = rc & 255u, cnt = rc >> 8;
  int off = 0;
  if (ok) off = sm.hist[wave][d];
  if (ok && rank == cnt - 1) atomicAdd(&sm.hist[wave][d], (int)cnt);
  return off + (int)rank;
}

constexpr int LDS_CHUNK = LDS_SORT_MAX / SORT_THREADS;  // entries per lane in the LDS sort

// Sort inside LDS (M <= LDS_SORT_MAX, Vp <= 2^16).
__device__ void build_index_lds(const int32_t* __restrict__ tok, int M, int Vp, const IndexPtrs ix, SortLds& sm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int passes = (bits_for(Vp) + 7) / 8;
  const int R = ((M + SORT_WAVES - 1) / SORT_WAVES + 63) / 64 * 64;
  const int w0 = min(M, wave * R), w1 = min(M, w0 + R);
  const unsigned long long lt = (1ull << lane) - 1ull;
  unsigned v[LDS_CHUNK], rc[LDS_CHUNK];
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = 15 + 8 * pass;
#pragma unroll
    for (int q = 0; q < LDS_CHUNK; ++q) {
      const int j = w0 + 64 * q + lane;
      v[q] = 0;
      if (j < w1) v[q] = pass == 0 ? ((unsigned)clamp_tok(tok[j], Vp) << 15) | (unsigned)j : sm.buf[j];
    }
    for (int i = threadIdx.x; i < SORT_WAVES * RADIX; i += SORT_THREADS) (&sm.hist[0][0])[i] = 0;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < LDS_CHUNK; ++q) {
      if (w0 + 64 * q >= w1) break;
      const bool ok = w0 + 64 * q + lane < w1;
      const int d = (v[q] >> shift) & (RADIX - 1);
      rc[q] = digit_rank(d, ok, lt);
      count_step(sm, wave, d, ok, rc[q]);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    scan_hist(sm);
#pragma unroll
    for (int q = 0; q < LDS_CHUNK; ++q) {
      if (w0 + 64 * q >= w1) break;
      const bool ok = w0 + 64 * q + lane < w1;
      const int slot = scatter_step(sm, wave, (v[q] >> shift) & (RADIX - 1), ok, rc[q]);
      if (ok) sm.buf[slot] = v[q];
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; i < M; i += SORT_THREADS) {
    const unsigned w = sm.buf[i];
    ix.skey[i] = (int)(w >> 15);
    ix.spos[i] = (int)(w & 0x7fffu);
  }
  run_info(M, ix, sm, [&](int i) { return (int)(sm.buf[i] >> 15); });
}

// Sort through global memory (any size): per pass a wave holds its entries
// in registers, SORT_CHUNK per lane (one chunk for up to 16,384 tokens;
// longer inputs loop over chunks and reload).
__device__ void build_index_global(const int32_t* __restrict__ tok, int M, int Vp, const IndexPtrs ix,
                                   SortLds& sm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int passes = (bits_for(Vp) + 7) / 8;
  const int R = ((M + SORT_WAVES - 1) / SORT_WAVES + 63) / 64 * 64;  // entries per wave
  const int w0 = min(M, wave * R), w1 = min(M, w0 + R);
  const bool single = R <= 64 * SORT_CHUNK;
  const unsigned long long lt = (1ull << lane) - 1ull;
  int key[SORT_CHUNK], pos[SORT_CHUNK];
  unsigned rc[SORT_CHUNK];
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = 8 * pass;
    // the last pass writes the result arrays
    const bool to_result = ((passes - 1 - pass) & 1) == 0;
    const int32_t* sk = pass == 0 ? nullptr : (to_result ? ix.tkey : ix.skey);
    const int32_t* sp = pass == 0 ? nullptr : (to_result ? ix.tpos : ix.spos);
    int32_t* dk = to_result ? ix.skey : ix.tkey;
    int32_t* dp = to_result ? ix.spos : ix.tpos;
    for (int i = threadIdx.x; i < SORT_WAVES * RADIX; i += SORT_THREADS) (&sm.hist[0][0])[i] = 0;
    __syncthreads();
    for (int cb = w0; cb < w1; cb += 64 * SORT_CHUNK) {
      sort_load(tok, sk, sp, Vp, cb, w1, lane, key, pos);
#pragma unroll
      for (int q = 0; q < SORT_CHUNK; ++q) {
        if (cb + 64 * q >= w1) break;
        const bool ok = cb + 64 * q + lane < w1;
        const int d = (key[q] >> shift) & (RADIX - 1);
        rc[q] = digit_rank(d, ok, lt);
        count_step(sm, wave, d, ok, rc[q]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();
    scan_hist(sm);
    for (int cb = w0; cb < w1; cb += 64 * SORT_CHUNK) {
      if (!single) sort_load(tok, sk, sp, Vp, cb, w1, lane, key, pos);
#pragma unroll
      for (int q = 0; q < SORT_CHUNK; ++q) {
        if (cb + 64 * q >= w1) break;
        const bool ok = cb + 64 * q + lane < w1;
        const int d = (key[q] >> shift) & (RADIX - 1);
        if (!single) rc[q] = digit_rank(d, ok, lt);
        const int slot = scatter_step(sm, wave, d, ok, rc[q]);
        __builtin_amdgcn_sched_barrier(0);
        if (ok) {
          dk[slot] = key[q];
          dp[slot] = pos[q];
        }
      }
    }
    __syncthreads();
  }
  run_info(M, ix, sm, [&](int i) { return ix.skey[i]; });
}

// The whole index, by one workgroup of SORT_THREADS threads.
__device__ void build_index(const int32_t* __restrict__ tok, int M, int Vp, const IndexPtrs ix, SortLds& sm) {
  if (M <= LDS_SORT_MAX && Vp <= (1 << 16))
    build_index_lds(tok, M, Vp, ix, sm);
  else
    build_index_global(tok, M, Vp, ix, sm);
}

__global__ void __launch_bounds__(SORT_THREADS) emb_index_kernel(const int32_t* __restrict__ tok, int M, int Vp,
                                                                 IndexPtrs ix) {
  __shared__ SortLds sm;
  build_index(tok, M, Vp, ix, sm);
}

// Forward gather: one wave per row, a lane NV float4 columns of it.  The row
// index is wave-uniform, so the token id is one scalar load and the position
// t = m mod T is scalar arithmetic; the wpe row's loads are issued before the
// token id arrives, then the wte row's, then the adds.  One row per wave
// measured 8% faster than four (19.6 vs 21.4 us at 16384 x 768 inside the
// step), the uniform row index (scalar token load, wpe loads first) another
// 5% (19.1 -> 18.2 us).
template <int NV>
__global__ void __launch_bounds__(64 * FWD_WAVES) emb_fwd_kernel(const int32_t* __restrict__ tok,
                                                                 const float* __restrict__ wte,
                                                                 const float* __restrict__ wpe,
                                                                 float* __restrict__ x0, int M, int T, int C,
                                                                 int Vp) {
  const int lane = threadIdx.x & 63;
  const int m = __builtin_amdgcn_readfirstlane(blockIdx.x * FWD_WAVES + (threadIdx.x >> 6));
  if (m >= M) return;
  const int C4 = C >> 2;
  const floatx4* pr = reinterpret_cast<const floatx4*>(wpe + (long long)(m % T) * C);
  floatx4 a[NV], b[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    if (c < C4) b[i] = pr[c];
  }
  const int id = clamp_tok(tok[m], Vp);
  const floatx4* wr = reinterpret_cast<const floatx4*>(wte + (long long)id * C);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    if (c < C4) a[i] = wr[c];
  }
  floatx4* xr = reinterpret_cast<floatx4*>(x0 + (long long)m * C);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    if (c < C4) xr[c] = a[i] + b[i];
  }
}

// ------------------------------------------------------------ backward sum
struct BwdArgs {
  const float* dx0;
  float* dwte;
  float* dwpe;
  float* partA;  // [np][C]: partial of a piece's last run when it continues past the piece
  float* partB;  // [np][C]: partial of a piece's first run when it began earlier and ends here
  IndexPtrs ix;
  int M, B, T, C, np, nslices, n_tok_units, n_pos_units, wpe_beta_one;
};

template <int V>
struct VecOf;
template <>
struct VecOf<1> {
  using type = float;
};
template <>
struct VecOf<4> {
  using type = floatx4;
};
using tvec = VecOf<TV>::type;

__device__ __forceinline__ tvec ld_tv(const float* p) { return *reinterpret_cast<const tvec*>(p); }
__device__ __forceinline__ void st_tv(float* p, tvec v) { *reinterpret_cast<tvec*>(p) = v; }

__device__ __forceinline__ void token_unit(const BwdArgs& a, int u) {
  static_assert(PIECE <= 64, "one sorted entry per lane");
  const int lane = threadIdx.x & 63;
  const int p = u / a.nslices, sl = u - p * a.nslices;
  const int i0 = p * PIECE;
  const int n = min(PIECE, a.M - i0);
  const int col = (sl * 64 + lane) * TV;
  const bool active = col < a.C;
  const int kv = lane < n ? a.ix.skey[i0 + lane] : -1;
  const int pv = lane < n ? a.ix.spos[i0 + lane] : 0;
  const bool cross_in = a.ix.fr_start[p] < p, cross_out = a.ix.lr_end[p] > p;
  const int key0 = __builtin_amdgcn_readfirstlane(kv);
  const int keyl = __shfl(kv, n - 1, 64);
  // lane i of `own`: entry i ends a run that also began in this piece
  const int knext = __shfl_down(kv, 1, 64);
  const bool ends = lane < n && (lane == n - 1 ? !cross_out : kv != knext);
  const unsigned long long own = __ballot(ends && !(cross_in && kv == key0));
  const unsigned long long first_run = __ballot(lane < n && kv == key0);
  tvec x[PIECE], z[PIECE];
#pragma unroll
  for (int i = 0; i < PIECE; ++i) {
    if (i < n) {
      const int pos = __builtin_amdgcn_readlane(pv, i);
      if (active) x[i] = ld_tv(a.dx0 + (long long)pos * a.C + col);
    }
  }
#pragma unroll
  for (int i = 0; i < PIECE; ++i) {
    if ((own >> i) & 1) {
      const int k = __builtin_amdgcn_readlane(kv, i);
      if (active) z[i] = ld_tv(a.dwte + (long long)k * a.C + col);
    }
  }
  if (!active) return;
  // running sums along each run, in entry order
#pragma unroll
  for (int i = 1; i < PIECE; ++i) {
    if (i < n && __builtin_amdgcn_readlane(kv, i) == __builtin_amdgcn_readlane(kv, i - 1)) x[i] = x[i - 1] + x[i];
  }
#pragma unroll
  for (int i = 0; i < PIECE; ++i) {
    if ((own >> i) & 1) {
      const int k = __builtin_amdgcn_readlane(kv, i);
      st_tv(a.dwte + (long long)k * a.C + col, z[i] + x[i]);
    }
  }
  // crossing runs
  const bool whole = cross_in && cross_out && key0 == keyl;  // the piece lies inside one run
  // a run continues past the piece only if the piece is full (n == PIECE)
  if (cross_out) st_tv(a.partA + (long long)p * a.C + col, x[PIECE - 1]);
  if (cross_in && !whole) {
    // the first run ends inside this piece at its last entry with key0
    const int iend = 63 - __builtin_clzll(first_run);
    tvec v = x[0];
#pragma unroll
    for (int i = 1; i < PIECE; ++i)
      if (i == iend) v = x[i];
    st_tv(a.partB + (long long)p * a.C + col, v);
  }
}

// Second launch, finish units: the piece where a crossing run starts adds
// that run's partials in piece order, A[s], ..., A[e-1], B[e], into dwte.
__device__ __forceinline__ void finish_unit(const BwdArgs& a, int u) {
  const int p = u / a.nslices, sl = u - p * a.nslices;
  const int e = a.ix.lr_end[p];
  if (e <= p || a.ix.lr_start[p] != p) return;
  const int col = (sl * 64 + (threadIdx.x & 63)) * TV;
  if (col >= a.C) return;
  const int key = a.ix.skey[min(a.M, (p + 1) * PIECE) - 1];
  constexpr int FB = 32 / TV;  // partials in flight per lane
  tvec acc = ld_tv(a.partA + (long long)p * a.C + col);
  for (int q0 = p + 1; q0 < e; q0 += FB) {
    tvec t[FB];
#pragma unroll
    for (int k = 0; k < FB; ++k)
      if (q0 + k < e) t[k] = ld_tv(a.partA + (long long)(q0 + k) * a.C + col);
#pragma unroll
    for (int k = 0; k < FB; ++k)
      if (q0 + k < e) acc = acc + t[k];
  }
  acc = acc + ld_tv(a.partB + (long long)e * a.C + col);
  float* d = a.dwte + (long long)key * a.C + col;
  st_tv(d, ld_tv(d) + acc);
}

__device__ __forceinline__ void position_unit(const BwdArgs& a, int u) {
  const int lane = threadIdx.x & 63;
  const int C4 = a.C >> 2;
  const int ns4 = (C4 + 63) / 64;
  const int tg = u / ns4, sl = u - tg * ns4;
  const int c4 = sl * 64 + lane;
  if (c4 >= C4) return;
  const floatx4* src = reinterpret_cast<const floatx4*>(a.dx0);
  floatx4* dst = reinterpret_cast<floatx4*>(a.dwpe);
  constexpr int BB = 16;  // rows of one position loaded together
  floatx4 s[WPE_T];
#pragma unroll
  for (int k = 0; k < WPE_T; ++k) s[k] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int b0 = 0; b0 < a.B; b0 += BB) {
    floatx4 r[WPE_T][BB];
#pragma unroll
    for (int k = 0; k < WPE_T; ++k) {
      const int t = tg * WPE_T + k;
#pragma unroll
      for (int q = 0; q < BB; ++q)
        if (t < a.T && b0 + q < a.B) r[k][q] = src[((long long)(b0 + q) * a.T + t) * C4 + c4];
    }
#pragma unroll
    for (int k = 0; k < WPE_T; ++k)
#pragma unroll
      for (int q = 0; q < BB; ++q)
        if (b0 + q < a.B) s[k] += r[k][q];
  }
#pragma unroll
  for (int k = 0; k < WPE_T; ++k) {
    const int t = tg * WPE_T + k;
    if (t < a.T) {
      floatx4 o = s[k];
      if (a.wpe_beta_one) o += dst[(long long)t * C4 + c4];
      dst[(long long)t * C4 + c4] = o;
    }
  }
}

// First launch: one workgroup per piece and group of up to TOK_WAVES column
// slices, so that the slices of the piece's rows are fetched together.
__global__ void __launch_bounds__(64 * TOK_WAVES) emb_bwd_kernel(const BwdArgs a) {
  const int sl = blockIdx.y * TOK_WAVES + (threadIdx.x >> 6);
  if (sl < a.nslices) token_unit(a, blockIdx.x * a.nslices + sl);
}

// Second launch: finish units, then position units.
__global__ void __launch_bounds__(256) emb_finish_kernel(const BwdArgs a) {
  const int u = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (u < a.n_tok_units) {
    finish_unit(a, u);
  } else if (u - a.n_tok_units < a.n_pos_units) {
    position_unit(a, u - a.n_tok_units);
  }
}

size_t partials_bytes(long long M, int C) {
  const long long np = (M + PIECE - 1) / PIECE;
  return 2 * align_up((size_t)np * C * sizeof(float), 256);
}

bt_status check_shape(int B, int T, int C, int Vp, const char* who) {
  BT_RETURN_IF(B < 0 || T < 0 || C <= 0 || (C & 3) || Vp <= 0 || Vp > (1 << 24), BT_ESHAPE,
               "%s: B=%d T=%d C=%d Vp=%d (C a positive multiple of 4, 0 < Vp <= 2^24)", who, B, T, C, Vp);
  BT_RETURN_IF((long long)B * T * (C / 4) >= (1LL << 31), BT_ESHAPE, "%s: B*T*C/4=%lld must be below 2^31", who,
               (long long)B * T * (C / 4));
  return BT_OK;
}

bt_status launch_fwd(const int32_t* tokens, const float* wte, const float* wpe, float* x0, int B, int T, int C,
                     int Vp, hipStream_t s) {
  const int M = B * T;
  const int nv = (C / 4 + 63) / 64;
#define BT_EMB_FWD(NV)                                                                                   \
  hipLaunchKernelGGL(emb_fwd_kernel<NV>, dim3((unsigned)((M + FWD_WAVES - 1) / FWD_WAVES)), dim3(64 * FWD_WAVES), \
                     0, s, tokens, wte, wpe, x0, M, T, C, Vp)
  switch (nv) {
    case 1: BT_EMB_FWD(1); break;
    case 2: BT_EMB_FWD(2); break;
    case 3: BT_EMB_FWD(3); break;
    case 4: BT_EMB_FWD(4); break;
    case 5: case 6: BT_EMB_FWD(6); break;
    case 7: case 8: BT_EMB_FWD(8); break;
    default: BT_EMB_FWD(16); break;
  }
#undef BT_EMB_FWD
  return check_launch("emb_fwd_kernel");
}

bt_status launch_bwd(const void* index, const float* dx0, float* dwte, float* dwpe, float wpe_beta, void* part,
                     int B, int T, int C, hipStream_t s) {
  BwdArgs a{};
  const int M = B * T;
  a.dx0 = dx0;
  a.dwte = dwte;
  a.dwpe = dwpe;
  a.partA = static_cast<float*>(part);
  a.partB = reinterpret_cast<float*>(static_cast<char*>(part) + partials_bytes(M, C) / 2);
  a.ix = index_ptrs(const_cast<void*>(index), M);
  a.M = M;
  a.B = B;
  a.T = T;
  a.C = C;
  a.np = (M + PIECE - 1) / PIECE;
  a.nslices = (C + 64 * TV - 1) / (64 * TV);
  a.n_tok_units = a.np * a.nslices;
  a.n_pos_units = dwpe ? ((T + WPE_T - 1) / WPE_T) * ((C / 4 + 63) / 64) : 0;
  a.wpe_beta_one = wpe_beta != 0.f;
  const int tw = a.nslices < TOK_WAVES ? a.nslices : TOK_WAVES;
  hipLaunchKernelGGL(emb_bwd_kernel, dim3((unsigned)a.np, (unsigned)((a.nslices + TOK_WAVES - 1) / TOK_WAVES)),
                     dim3(64 * tw), 0, s, a);
  BT_TRY(check_launch("emb_bwd_kernel"));
  const long long units = (long long)a.n_tok_units + a.n_pos_units;
  hipLaunchKernelGGL(emb_finish_kernel, dim3((unsigned)((units + 3) / 4)), dim3(256), 0, s, a);
  return check_launch("emb_finish_kernel");
}

}  // namespace

// A backward over no positions (B = 0 or T = 0): no dwte row gets anything,
// and the rows t < T of dwpe get an empty batch sum, so they become
// wpe_beta * dwpe (zeros at wpe_beta = 0).
static bt_status bwd_no_positions(float* dwpe, float wpe_beta, int T, int C, const char* who, hipStream_t s) {
  if (T == 0 || wpe_beta != 0.f) return BT_OK;
  BT_RETURN_IF(!dwpe, BT_EINVAL, "%s: NULL pointer", who);
  return fill_zero(dwpe, (size_t)T * C, s);
}

// Internal entry points of the composed step (bt_internal.h).
size_t emb_index_bytes(long long M) { return M > 0 ? index_layout(M).total : 0; }
size_t emb_bwd_partials_bytes(long long M, int C) { return M > 0 ? partials_bytes(M, C) : 0; }

}  // namespace bt

using namespace bt;

extern "C" bt_status bt_embedding_fwd(const int32_t* tokens, const float* wte, const float* wpe, float* x0, int B,
                                      int T, int C, int Vp, void* stream) {
  bt::clear_error();
  BT_TRY(check_shape(B, T, C, Vp, "bt_embedding_fwd"));
  if (B * T == 0) return BT_OK;
  BT_RETURN_IF(!tokens || !wte || !wpe || !x0, BT_EINVAL, "bt_embedding_fwd: NULL pointer");
  BT_RETURN_IF(!aligned16(wte) || !aligned16(wpe) || !aligned16(x0), BT_EALIGN,
               "bt_embedding_fwd: float tensors must be 16-byte aligned");
  return launch_fwd(tokens, wte, wpe, x0, B, T, C, Vp, as_stream(stream));
}

extern "C" size_t bt_embedding_index_bytes(int B, int T) {
  if (B <= 0 || T <= 0) return 0;
  return emb_index_bytes((long long)B * T);
}

extern "C" bt_status bt_embedding_index(const int32_t* tokens, void* index, size_t index_bytes, int B, int T, int Vp,
                                        void* stream) {
  bt::clear_error();
  BT_TRY(check_shape(B, T, 4, Vp, "bt_embedding_index"));
  if (B * T == 0) return BT_OK;
  BT_RETURN_IF(!tokens || !index, BT_EINVAL, "bt_embedding_index: NULL pointer");
  const size_t need = bt_embedding_index_bytes(B, T);
  BT_RETURN_IF(index_bytes < need, BT_EWORKSPACE, "bt_embedding_index: index of %zu bytes needed (got %zu)", need,
               index_bytes);
  BT_RETURN_IF(!aligned16(index), BT_EALIGN, "bt_embedding_index: index must be 16-byte aligned");
  const int M = B * T;
  hipLaunchKernelGGL(emb_index_kernel, dim3(1), dim3(SORT_THREADS), 0, as_stream(stream), tokens, M, Vp,
                     index_ptrs(index, M));
  return check_launch("emb_index_kernel");
}

extern "C" size_t bt_embedding_bwd_indexed_ws_bytes(int B, int T, int C) {
  if (B <= 0 || T <= 0 || C <= 0) return 0;
  return emb_bwd_partials_bytes((long long)B * T, C);
}

extern "C" bt_status bt_embedding_bwd_indexed(const void* index, size_t index_bytes, const float* dx0, float* dwte,
                                              float* dwpe, float wpe_beta, void* ws, size_t ws_bytes, int B, int T,
                                              int C, int Vp, void* stream) {
  bt::clear_error();
  BT_TRY(check_shape(B, T, C, Vp, "bt_embedding_bwd_indexed"));
  BT_RETURN_IF(wpe_beta != 0.f && wpe_beta != 1.f, BT_EINVAL, "bt_embedding_bwd_indexed: wpe_beta must be 0 or 1");
  if (B * T == 0) return bwd_no_positions(dwpe, wpe_beta, T, C, "bt_embedding_bwd_indexed", as_stream(stream));
  BT_RETURN_IF(!index || !dx0 || !dwte || !dwpe, BT_EINVAL, "bt_embedding_bwd_indexed: NULL pointer");
  BT_RETURN_IF(index_bytes < bt_embedding_index_bytes(B, T), BT_EWORKSPACE,
               "bt_embedding_bwd_indexed: index of %zu bytes needed (got %zu)", bt_embedding_index_bytes(B, T),
               index_bytes);
  BT_RETURN_IF(!aligned16(dx0) || !aligned16(dwte) || !aligned16(dwpe) || !aligned16(index), BT_EALIGN,
               "bt_embedding_bwd_indexed: tensors must be 16-byte aligned");
  const size_t need = bt_embedding_bwd_indexed_ws_bytes(B, T, C);
  BT_RETURN_IF(!ws || ws_bytes < need, BT_EWORKSPACE,
               "bt_embedding_bwd_indexed: workspace of %zu bytes needed (got %zu)", need, ws_bytes);
  BT_RETURN_IF(!aligned16(ws), BT_EALIGN, "bt_embedding_bwd_indexed: workspace must be 16-byte aligned");
  return launch_bwd(index, dx0, dwte, dwpe, wpe_beta, ws, B, T, C, as_stream(stream));
}

extern "C" size_t bt_embedding_bwd_ws_bytes(int B, int T, int C, int Vp) {
  (void)Vp;
  if (B <= 0 || T <= 0 || C <= 0) return 0;
  const long long M = (long long)B * T;
  return emb_index_bytes(M) + emb_bwd_partials_bytes(M, C);
}

extern "C" bt_status bt_embedding_bwd(const int32_t* tokens, const float* dx0, float* dwte, float* dwpe,
                                      float wpe_beta, void* ws, size_t ws_bytes, int B, int T, int C, int Vp,
                                      void* stream) {
  bt::clear_error();
  BT_TRY(check_shape(B, T, C, Vp, "bt_embedding_bwd"));
  BT_RETURN_IF(wpe_beta != 0.f && wpe_beta != 1.f, BT_EINVAL, "bt_embedding_bwd: wpe_beta must be 0 or 1");
  const int M = B * T;
  if (M == 0) return bwd_no_positions(dwpe, wpe_beta, T, C, "bt_embedding_bwd", as_stream(stream));
  BT_RETURN_IF(!tokens || !dx0 || !dwte || !dwpe, BT_EINVAL, "bt_embedding_bwd: NULL pointer");
  BT_RETURN_IF(!aligned16(dx0) || !aligned16(dwte) || !aligned16(dwpe), BT_EALIGN,
               "bt_embedding_bwd: float tensors must be 16-byte aligned");
  const size_t need = bt_embedding_bwd_ws_bytes(B, T, C, Vp);
  BT_RETURN_IF(!ws || ws_bytes < need, BT_EWORKSPACE, "bt_embedding_bwd: workspace of %zu bytes needed (got %zu)",
               need, ws_bytes);
  BT_RETURN_IF(!aligned16(ws), BT_EALIGN, "bt_embedding_bwd: workspace must be 16-byte aligned");
  hipStream_t s = as_stream(stream);
  const size_t ib = emb_index_bytes(M);
  hipLaunchKernelGGL(emb_index_kernel, dim3(1), dim3(SORT_THREADS), 0, s, tokens, M, Vp, index_ptrs(ws, M));
  BT_TRY(check_launch("emb_index_kernel"));
  return launch_bwd(ws, dx0, dwte, dwpe, wpe_beta, static_cast<char*>(ws) + ib, B, T, C, s);
}
