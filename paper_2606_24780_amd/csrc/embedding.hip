// Token + position embeddings with the token table tied to the LM head
// (GPT-2 architecture figure: weight-tied embeddings, learned positions).
//
// Forward: x0[b, t] = wte[tok[b, t]] + wpe[t], one float4 per thread.
// Backward (deterministic, no float atomics):
//  * dwpe[t] = beta dwpe[t] + sum_b dx0[b, t] in batch order;
//  * dwte: positions are sorted by (token, position) with a device radix
//    sort of unique 32/64-bit keys, then each token's rows are summed in
//    position order.  The sorted list is cut into chunks of 32 entries; a
//    token whose run lies inside one chunk is added to dwte directly by that
//    chunk, a run that crosses chunk boundaries is summed chunk by chunk into
//    partials which the chunk where the run ends adds up in order.  The heavy
//    head of the Zipf token distribution (about 14% of positions for id 0)
//    is therefore spread over many blocks instead of one.
#include <rocprim/device/device_radix_sort.hpp>

#include "bt_internal.h"

namespace bt {
namespace {

constexpr int CHUNK = 32;

__global__ void __launch_bounds__(256) emb_fwd_kernel(const int32_t* __restrict__ tok, const float* __restrict__ wte,
                                                      const float* __restrict__ wpe, float* __restrict__ x0,
                                                      int M, int T, int C, int Vp) {
  const int C4 = C >> 2;
  const long long n4 = (long long)M * C4;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < n4;
       e += (long long)gridDim.x * blockDim.x) {
    const int m = (int)(e / C4), c = (int)(e - (long long)m * C4);
    int id = tok[m];
    id = id < 0 ? 0 : (id >= Vp ? Vp - 1 : id);
    const int t = m % T;
    const floatx4 a = reinterpret_cast<const floatx4*>(wte + (long long)id * C)[c];
    const floatx4 b = reinterpret_cast<const floatx4*>(wpe + (long long)t * C)[c];
    reinterpret_cast<floatx4*>(x0 + (long long)m * C)[c] = a + b;
  }
}

__global__ void __launch_bounds__(256) wpe_bwd_kernel(const float* __restrict__ dx0, float* __restrict__ dwpe,
                                                      int B, int T, int C, float beta) {
  const int C4 = C >> 2;
  const long long n4 = (long long)T * C4;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < n4;
       e += (long long)gridDim.x * blockDim.x) {
    const int t = (int)(e / C4), c = (int)(e - (long long)t * C4);
    floatx4 s = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int b = 0; b < B; ++b) s += reinterpret_cast<const floatx4*>(dx0 + ((long long)b * T + t) * C)[c];
    floatx4* d = reinterpret_cast<floatx4*>(dwpe + (long long)t * C) + c;
    if (beta != 0.f) s += *d;
    *d = s;
  }
}

template <typename K>
__global__ void __launch_bounds__(256) make_keys(const int32_t* __restrict__ tok, K* __restrict__ keys, int M,
                                                 int pos_bits, int Vp) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  int id = tok[m];
  id = id < 0 ? 0 : (id >= Vp ? Vp - 1 : id);
  keys[m] = ((K)id << pos_bits) | (K)m;
}

// Chunk pass.  part holds, per chunk, [first-run partial | last-run partial].
template <typename K>
__global__ void __launch_bounds__(256) wte_chunk_kernel(const K* __restrict__ keys, const float* __restrict__ dx0,
                                                        float* __restrict__ dwte, float* __restrict__ part, int M,
                                                        int C, int pos_bits) {
  const int ch = blockIdx.x;
  const int lo = ch * CHUNK, hi = min(M, lo + CHUNK);
  const K mask = ((K)1 << pos_bits) - 1;
  __shared__ int s_tok[CHUNK + 2];
  __shared__ int s_pos[CHUNK];
  for (int i = threadIdx.x; i < hi - lo; i += blockDim.x) {
    const K k = keys[lo + i];
    s_tok[i + 1] = (int)(k >> pos_bits);
    s_pos[i] = (int)(k & mask);
  }
  if (threadIdx.x == 0) {
    s_tok[0] = lo > 0 ? (int)(keys[lo - 1] >> pos_bits) : -1;
    s_tok[hi - lo + 1] = hi < M ? (int)(keys[hi] >> pos_bits) : -1;
  }
  __syncthreads();
  const int C4 = C >> 2;
  const int n = hi - lo;
  for (int c = threadIdx.x; c < C4; c += blockDim.x) {
    floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
    bool run_started_here = s_tok[1] != s_tok[0];
    for (int i = 0; i < n; ++i) {
      acc += reinterpret_cast<const floatx4*>(dx0 + (long long)s_pos[i] * C)[c];
      const bool run_ends = s_tok[i + 2] != s_tok[i + 1];
      if (run_ends || i == n - 1) {
        const int tk = s_tok[i + 1];
        if (run_started_here && run_ends) {
          floatx4* d = reinterpret_cast<floatx4*>(dwte + (long long)tk * C) + c;
          *d += acc;  // the whole run lies in this chunk: sole writer of this row
        } else if (!run_started_here) {
          reinterpret_cast<floatx4*>(part + (long long)ch * 2 * C)[c] = acc;       // continues from before
        } else {
          reinterpret_cast<floatx4*>(part + (long long)ch * 2 * C + C)[c] = acc;   // continues past the end
        }
        acc = floatx4{0.f, 0.f, 0.f, 0.f};
        run_started_here = true;
      }
    }
  }
}

// Finish runs that cross chunk boundaries: chunk ch handles the run that
// entered it from the previous chunk and ends inside it.
template <typename K>
__global__ void __launch_bounds__(256) wte_span_kernel(const K* __restrict__ keys, const float* __restrict__ part,
                                                       float* __restrict__ dwte, int M, int C, int pos_bits) {
  const int ch = blockIdx.x;
  const int lo = ch * CHUNK, hi = min(M, lo + CHUNK);
  if (lo == 0) return;
  const int tk = (int)(keys[lo] >> pos_bits);
  if ((int)(keys[lo - 1] >> pos_bits) != tk) return;           // run starts here: not a crossing run
  if ((int)(keys[hi - 1] >> pos_bits) == tk && hi < M && (int)(keys[hi] >> pos_bits) == tk)
    return;                                                     // run continues past this chunk
  // walk back to the chunk where the run starts
  int s = ch - 1;
  while (s > 0 && (int)(keys[s * CHUNK - 1] >> pos_bits) == tk && (int)(keys[s * CHUNK] >> pos_bits) == tk) --s;
  // the run starts inside chunk s and runs past its end: chunk s stored it as
  // its last-run partial; chunks s+1..ch-1 are covered whole (first-run
  // partials) and chunk ch holds the run's tail (first-run partial)
  const int C4 = C >> 2;
  for (int c = threadIdx.x; c < C4; c += blockDim.x) {
    floatx4 acc = reinterpret_cast<const floatx4*>(part + (long long)s * 2 * C + C)[c];
    for (int k = s + 1; k < ch; ++k) acc += reinterpret_cast<const floatx4*>(part + (long long)k * 2 * C)[c];
    acc += reinterpret_cast<const floatx4*>(part + (long long)ch * 2 * C)[c];
    floatx4* d = reinterpret_cast<floatx4*>(dwte + (long long)tk * C) + c;
    *d += acc;
  }
}

int bits_for(long long n) {
  int b = 0;
  while ((1LL << b) < n) ++b;
  return b < 1 ? 1 : b;
}

template <typename K>
size_t sort_temp_bytes(int M, unsigned end_bit) {
  size_t bytes = 0;
  if (rocprim::radix_sort_keys(nullptr, bytes, (K*)nullptr, (K*)nullptr, (size_t)M, 0u, end_bit) != hipSuccess)
    return 0;
  return bytes;
}

struct EmbWs {
  size_t keys_off, sorted_off, part_off, temp_off, temp_bytes, total;
};

int bits_for(long long n);

template <typename K>
EmbWs emb_layout(int M, int C, int Vp) {
  EmbWs w;
  const size_t nch = (M + CHUNK - 1) / CHUNK;
  w.keys_off = 0;
  w.sorted_off = align_up(sizeof(K) * M, 256);
  w.part_off = w.sorted_off + align_up(sizeof(K) * M, 256);
  w.temp_off = w.part_off + align_up(nch * 2 * C * sizeof(float), 256);
  w.temp_bytes = sort_temp_bytes<K>(M, (unsigned)(bits_for(M) + bits_for(Vp)));
  w.total = w.temp_off + align_up(w.temp_bytes, 256);
  return w;
}

bool use64(int M, int Vp) { return bits_for(M) + bits_for(Vp) > 32; }

template <typename K>
bt_status wte_bwd(const int32_t* tok, const float* dx0, float* dwte, char* ws, int M, int C, int Vp,
                  hipStream_t s) {
  const EmbWs w = emb_layout<K>(M, C, Vp);
  const int pos_bits = bits_for(M);
  K* keys = reinterpret_cast<K*>(ws + w.keys_off);
  K* sorted = reinterpret_cast<K*>(ws + w.sorted_off);
  float* part = reinterpret_cast<float*>(ws + w.part_off);
  hipLaunchKernelGGL(make_keys<K>, dim3((M + 255) / 256), dim3(256), 0, s, tok, keys, M, pos_bits, Vp);
  BT_TRY(check_launch("make_keys"));
  size_t tb = w.temp_bytes;
  const unsigned end_bit = (unsigned)(pos_bits + bits_for(Vp));
  BT_CHECK_HIP(rocprim::radix_sort_keys(ws + w.temp_off, tb, keys, sorted, (size_t)M, 0u, end_bit, s));
  const int nch = (M + CHUNK - 1) / CHUNK;
  hipLaunchKernelGGL(wte_chunk_kernel<K>, dim3(nch), dim3(256), 0, s, sorted, dx0, dwte, part, M, C, pos_bits);
  BT_TRY(check_launch("wte_chunk_kernel"));
  hipLaunchKernelGGL(wte_span_kernel<K>, dim3(nch), dim3(256), 0, s, sorted, part, dwte, M, C, pos_bits);
  return check_launch("wte_span_kernel");
}

}  // namespace
}  // namespace bt

using namespace bt;

extern "C" bt_status bt_embedding_fwd(const int32_t* tokens, const float* wte, const float* wpe, float* x0, int B,
                                      int T, int C, int Vp, void* stream) {
  BT_RETURN_IF(B < 0 || T < 0 || C <= 0 || (C & 3) || Vp <= 0, BT_ESHAPE,
               "bt_embedding_fwd: B=%d T=%d C=%d Vp=%d", B, T, C, Vp);
  const int M = B * T;
  if (M == 0) return BT_OK;
  BT_RETURN_IF(!tokens || !wte || !wpe || !x0, BT_EINVAL, "bt_embedding_fwd: NULL pointer");
  BT_RETURN_IF(!aligned16(wte) || !aligned16(wpe) || !aligned16(x0), BT_EALIGN,
               "bt_embedding_fwd: float tensors must be 16-byte aligned");
  const long long n4 = (long long)M * (C / 4);
  long long nb = (n4 + 255) / 256;
  if (nb > 2048) nb = 2048;
  hipLaunchKernelGGL(emb_fwd_kernel, dim3((unsigned)nb), dim3(256), 0, as_stream(stream), tokens, wte, wpe, x0, M, T,
                     C, Vp);
  return check_launch("emb_fwd_kernel");
}

extern "C" size_t bt_embedding_bwd_ws_bytes(int B, int T, int C, int Vp) {
  const long long M = (long long)B * T;
  if (M <= 0 || C <= 0) return 0;
  return use64((int)M, Vp) ? emb_layout<unsigned long long>((int)M, C, Vp).total
                           : emb_layout<unsigned int>((int)M, C, Vp).total;
}

extern "C" bt_status bt_embedding_bwd(const int32_t* tokens, const float* dx0, float* dwte, float* dwpe,
                                      float wpe_beta, void* ws, size_t ws_bytes, int B, int T, int C, int Vp,
                                      void* stream) {
  BT_RETURN_IF(B < 0 || T < 0 || C <= 0 || (C & 3) || Vp <= 0, BT_ESHAPE,
               "bt_embedding_bwd: B=%d T=%d C=%d Vp=%d", B, T, C, Vp);
  BT_RETURN_IF(wpe_beta != 0.f && wpe_beta != 1.f, BT_EINVAL, "bt_embedding_bwd: wpe_beta must be 0 or 1");
  const int M = B * T;
  if (M == 0) return BT_OK;
  BT_RETURN_IF(!tokens || !dx0 || !dwte || !dwpe, BT_EINVAL, "bt_embedding_bwd: NULL pointer");
  BT_RETURN_IF(!aligned16(dx0) || !aligned16(dwte) || !aligned16(dwpe), BT_EALIGN,
               "bt_embedding_bwd: float tensors must be 16-byte aligned");
  const size_t need = bt_embedding_bwd_ws_bytes(B, T, C, Vp);
  BT_RETURN_IF(!ws || ws_bytes < need, BT_EWORKSPACE, "bt_embedding_bwd: workspace of %zu bytes needed (got %zu)",
               need, ws_bytes);
  BT_RETURN_IF(!aligned16(ws), BT_EALIGN, "bt_embedding_bwd: workspace must be 16-byte aligned");
  hipStream_t s = as_stream(stream);
  const long long n4 = (long long)T * (C / 4);
  long long nb = (n4 + 255) / 256;
  if (nb > 2048) nb = 2048;
  hipLaunchKernelGGL(wpe_bwd_kernel, dim3((unsigned)nb), dim3(256), 0, s, dx0, dwpe, B, T, C, wpe_beta);
  BT_TRY(check_launch("wpe_bwd_kernel"));
  if (use64(M, Vp))
    return wte_bwd<unsigned long long>(tokens, dx0, dwte, static_cast<char*>(ws), M, C, Vp, s);
  return wte_bwd<unsigned int>(tokens, dx0, dwte, static_cast<char*>(ws), M, C, Vp, s);
}
