// Composed GPT-2 training step on one GPU's data-parallel shard.
//
// One micro-step of the data-parallel training-step algorithm (forward,
// cross-entropy against the target, backward) followed, once per step, by
// global-norm clipping and the fused AdamW update.  Model: pre-LN GPT-2
// decoder with tied token embedding / LM head and learned positions (GPT-2
// architecture figure, hyper-parameter table).
//
// Everything is enqueued on the context's stream (about 20 launches per layer
// plus a few); the only host synchronisation is the final loss read in
// bt_gpt2_train_step.  Activations saved for the backward live in the
// caller's workspace, laid out once per context for max_B x max_T tokens.
#include <cmath>
#include <vector>

#include "bt_internal.h"

namespace bt {
bt_status launch_loss_sum(const float* rows, int n, float scale, int accumulate, float* d_loss, hipStream_t s);
}

using namespace bt;

namespace {

// element offsets of the named tensors in the flat arena
struct LayerOffs {
  size_t Wqkv, Wo, Wfc, Wfp, ln1g, ln1b, bqkv, bo, ln2g, ln2b, bfc, bfp;
};
struct ParamOffs {
  size_t wte, wpe, lnfg, lnfb, total, n_decay;
  std::vector<LayerOffs> layer;
  std::vector<size_t> all;  // every tensor start in canonical order + total
};

ParamOffs param_offsets(const bt_gpt2_config& c) {
  ParamOffs o;
  const size_t C = c.C, F = 4 * (size_t)c.C;
  size_t off = 0;
  auto take = [&](size_t n) {
    o.all.push_back(off);
    size_t r = off;
    off += n;
    return r;
  };
  o.layer.resize(c.L);
  o.wte = take((size_t)c.Vp * C);
  o.wpe = take((size_t)c.max_T * C);
  for (int l = 0; l < c.L; ++l) {
    o.layer[l].Wqkv = take(C * 3 * C);
    o.layer[l].Wo = take(C * C);
    o.layer[l].Wfc = take(C * F);
    o.layer[l].Wfp = take(F * C);
  }
  o.n_decay = off;
  for (int l = 0; l < c.L; ++l) {
    o.layer[l].ln1g = take(C);
    o.layer[l].ln1b = take(C);
    o.layer[l].bqkv = take(3 * C);
    o.layer[l].bo = take(C);
    o.layer[l].ln2g = take(C);
    o.layer[l].ln2b = take(C);
    o.layer[l].bfc = take(F);
    o.layer[l].bfp = take(C);
  }
  o.lnfg = take(C);
  o.lnfb = take(C);
  o.total = off;
  o.all.push_back(off);
  return o;
}

bt_status check_config(const bt_gpt2_config* c) {
  BT_RETURN_IF(!c, BT_EINVAL, "gpt2: config is NULL");
  BT_RETURN_IF(c->L < 1 || c->H < 1 || c->C < 4 || c->C % c->H || (c->C & 3), BT_ESHAPE,
               "gpt2: bad model shape L=%d H=%d C=%d", c->L, c->H, c->C);
  const int hd = c->C / c->H;
  BT_RETURN_IF(hd > 128 || (hd & 3), BT_ESHAPE, "gpt2: head dim %d unsupported (multiple of 4, <= 128)", hd);
  BT_RETURN_IF(c->C > 4096, BT_ESHAPE, "gpt2: C=%d > 4096 unsupported", c->C);
  BT_RETURN_IF(c->V < 1 || c->Vp < c->V || (c->Vp & 3), BT_ESHAPE, "gpt2: V=%d Vp=%d (Vp >= V, multiple of 4)",
               c->V, c->Vp);
  BT_RETURN_IF(c->max_T < 1, BT_ESHAPE, "gpt2: max_T=%d", c->max_T);
  BT_RETURN_IF(!(c->ln_eps >= 0.f), BT_EINVAL, "gpt2: ln_eps must be >= 0");
  return BT_OK;
}

// Workspace layout for M = max_B * max_T tokens.
struct Layout {
  size_t res, ln1, mu1, rs1, qkv, att, lse, xmid, ln2, mu2, rs2, h, g;  // per-layer bases
  size_t per_layer;                                                      // stride between layers
  size_t resL, lnf, muf, rsf, logits, loss_rows, lse_rows;
  size_t dres, dbig, dsmall;
  size_t ln_part, ln_part_slab;  // LayerNorm-backward partial rows: 2L+1 slabs of ln_part_slab floats
  size_t emb_index;              // token index built by the embedding forward, read by its backward
  size_t scalars;  // [loss, norm, coef, pad]
  size_t scratch, scratch_bytes;
  size_t total;
};

size_t scratch_need(const bt_gpt2_config& c, int B, int T) {
  const int M = B * T, C = c.C, F = 4 * c.C;
  size_t s = 0;
  auto mx = [&](size_t v) { s = v > s ? v : s; };
  // every product of the step may be split along K (an epilogue then runs in
  // the reduction); the split count depends on the token count, so cover
  // every call size <= M
  for (int m = M; m >= 1; m = m > 1 ? (m + 1) / 2 : 0) {
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_N, m, 3 * C, C, BT_EPI_BIAS));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_N, m, C, C, BT_EPI_BIAS));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_N, m, F, C, BT_EPI_BIAS_GELU));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_N, m, C, F, BT_EPI_BIAS));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_T, m, F, C, BT_EPI_DGELU));
    mx(bt_gemm_ws_bytes(BT_OP_T, BT_OP_N, C, 3 * C, m, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_T, BT_OP_N, C, C, m, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_T, BT_OP_N, C, F, m, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_T, BT_OP_N, F, C, m, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_T, BT_OP_N, c.Vp, C, m, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_N, m, C, c.Vp, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_T, m, c.Vp, C, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_T, m, C, 3 * C, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_T, m, C, C, BT_EPI_NONE));
    mx(bt_gemm_ws_bytes(BT_OP_N, BT_OP_T, m, C, F, BT_EPI_NONE));
    if (m == 1) break;
  }
  mx(bt_attention_bwd_ws_bytes(B, T, c.H, C / c.H));
  mx(bt_layernorm_bwd_ws_bytes(M, C));
  mx(bt_colsum_ws_bytes(M, F > 3 * C ? F : 3 * C));
  mx(emb_bwd_partials_bytes((long long)M, C));
  mx(bt_grad_norm_ws_bytes(param_offsets(c).total));
  return align_up(s, 256);
}

Layout make_layout(const bt_gpt2_config& c, int B, int T) {
  Layout o{};
  const size_t M = (size_t)B * T, C = c.C, F = 4 * (size_t)c.C, H = c.H;
  size_t off = 0;
  auto take = [&](size_t floats) {
    size_t r = off;
    off += align_up(floats * sizeof(float), 256);
    return r;
  };
  const size_t l0 = off;
  o.res = take(M * C);
  o.ln1 = take(M * C);
  o.mu1 = take(M);
  o.rs1 = take(M);
  o.qkv = take(M * 3 * C);
  o.att = take(M * C);
  o.lse = take(M * H);
  o.xmid = take(M * C);
  o.ln2 = take(M * C);
  o.mu2 = take(M);
  o.rs2 = take(M);
  o.h = take(M * F);
  o.g = take(M * F);
  o.per_layer = off - l0;
  off = l0 + o.per_layer * c.L;
  o.resL = take(M * C);
  o.lnf = take(M * C);
  o.muf = take(M);
  o.rsf = take(M);
  o.logits = take(M * (size_t)c.Vp);
  o.loss_rows = take(M);
  o.lse_rows = take(M);
  o.dres = take(M * C);
  o.dbig = take(M * (F > 3 * C ? F : 3 * C));
  o.dsmall = take(M * C);
  o.ln_part_slab = align_up((size_t)ln_bwd_partial_rows((int)M, (int)C) * 2 * C, 64);
  o.ln_part = take(o.ln_part_slab * (2 * (size_t)c.L + 1));
  o.scalars = take(64);
  o.emb_index = off;
  off += align_up(emb_index_bytes((long long)M), 256);
  o.scratch_bytes = scratch_need(c, B, T);
  o.scratch = off;
  off += o.scratch_bytes;
  o.total = off;
  return o;
}

}  // namespace

namespace {

struct ProfRec {
  int cls;
  double flops, bytes;
  hipEvent_t a, b;
};

struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<ProfRec> pending;
  bt_kernel_stat stats[BT_PROF_NCLASSES] = {};
  // end event of the previous profiled call when nothing has been enqueued
  // on the stream since: the next call starts from it (one record per call)
  hipEvent_t tail = nullptr;
};

}  // namespace

struct bt_gpt2_ctx {
  bt_gpt2_config cfg;
  char* ws;
  size_t ws_bytes;
  int max_B, max_T;
  hipStream_t stream;
  // the embedding backward's token index is built on a second stream while
  // the forward runs (fork after the caller's prior work, join before the
  // embedding backward)
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_index = nullptr;
  int t;
  ParamOffs po;
  Layout lay;
  Profiler prof;
};

namespace {

// Accumulate finished event pairs (the stream must have been synchronised).
bt_status prof_flush(bt_gpt2_ctx* c) {
  for (const ProfRec& r : c->prof.pending) {
    float ms = 0.f;
    BT_CHECK_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    bt_kernel_stat& s = c->prof.stats[r.cls];
    s.launches += 1;
    s.ms += ms;
    s.flops += r.flops;
    s.bytes += r.bytes;
  }
  c->prof.pending.clear();
  c->prof.used = 0;
  c->prof.tail = nullptr;
  return BT_OK;
}

// Work not bracketed by a profiled call was (or may have been) enqueued: the
// next profiled call records its own start event.
void prof_break(bt_gpt2_ctx* c) { c->prof.tail = nullptr; }

// Brackets one library call with events when profiling is on.  Back-to-back
// calls share the event between them, so a step records one event per call.
struct ProfScope {
  bt_gpt2_ctx* c;
  ProfRec rec;
  bool active = false;
  ProfScope(bt_gpt2_ctx* ctx, int cls, double flops, double bytes) : c(ctx) {
    if (!c->prof.on) return;
    if (c->prof.used + 2 > c->prof.pool.size()) {
      if (hipStreamSynchronize(c->stream) != hipSuccess || prof_flush(c) != BT_OK) return;
    }
    rec = ProfRec{cls, flops, bytes, c->prof.tail, nullptr};
    if (!rec.a) {
      rec.a = c->prof.pool[c->prof.used++];
      if (hipEventRecord(rec.a, c->stream) != hipSuccess) {
        c->prof.tail = nullptr;
        return;
      }
    }
    rec.b = c->prof.pool[c->prof.used++];
    active = true;
  }
  ~ProfScope() {
    if (!active) return;
    if (hipEventRecord(rec.b, c->stream) == hipSuccess) {
      c->prof.pending.push_back(rec);
      c->prof.tail = rec.b;
    } else {
      c->prof.tail = nullptr;
    }
  }
};

}  // namespace

#define BT_PROF(cls, flops, bytes, call)                     \
  do {                                                       \
    ProfScope _ps(ctx, (cls), (double)(flops), (double)(bytes)); \
    BT_TRY(call);                                            \
  } while (0)

extern "C" bt_status bt_gpt2_profile_enable(bt_gpt2_ctx* ctx, int enable) {
  bt::clear_error();
  BT_RETURN_IF(!ctx, BT_EINVAL, "bt_gpt2_profile_enable: ctx is NULL");
  if (enable && ctx->prof.pool.empty()) {
    // Timing-only events: without the system-scope fence an event record
    // costs no cache writeback / invalidate (with it, ~4 us of GPU time per
    // record, ~1.9 ms per GPT-2 124M step).  Elapsed times are read only
    // after the stream has synchronised.  16384 events cover ~35 steps
    // before the pool is flushed (a stream synchronisation).
    ctx->prof.pool.resize(16384);
    for (auto& e : ctx->prof.pool) BT_CHECK_HIP(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
  }
  ctx->prof.on = enable != 0;
  return BT_OK;
}

extern "C" bt_status bt_gpt2_profile_read(bt_gpt2_ctx* ctx, bt_kernel_stat* out, int reset) {
  bt::clear_error();
  BT_RETURN_IF(!ctx || !out, BT_EINVAL, "bt_gpt2_profile_read: NULL pointer");
  BT_CHECK_HIP(hipStreamSynchronize(ctx->stream));
  BT_TRY(prof_flush(ctx));
  for (int i = 0; i < BT_PROF_NCLASSES; ++i) out[i] = ctx->prof.stats[i];
  if (reset)
    for (auto& s : ctx->prof.stats) s = bt_kernel_stat{};
  return BT_OK;
}

extern "C" size_t bt_gpt2_num_params(const bt_gpt2_config* cfg) {
  if (check_config(cfg) != BT_OK) return 0;
  return param_offsets(*cfg).total;
}

extern "C" size_t bt_gpt2_num_decay_params(const bt_gpt2_config* cfg) {
  if (check_config(cfg) != BT_OK) return 0;
  return param_offsets(*cfg).n_decay;
}

extern "C" bt_status bt_gpt2_param_offsets(const bt_gpt2_config* cfg, size_t* offsets, int* n_tensors) {
  bt::clear_error();
  BT_TRY(check_config(cfg));
  BT_RETURN_IF(!n_tensors, BT_EINVAL, "bt_gpt2_param_offsets: n_tensors is NULL");
  const ParamOffs po = param_offsets(*cfg);
  *n_tensors = (int)po.all.size() - 1;
  if (offsets)
    for (size_t i = 0; i < po.all.size(); ++i) offsets[i] = po.all[i];
  return BT_OK;
}

extern "C" size_t bt_gpt2_workspace_bytes(const bt_gpt2_config* cfg, int max_B, int max_T) {
  if (check_config(cfg) != BT_OK || max_B < 1 || max_T < 1) return 0;
  return make_layout(*cfg, max_B, max_T).total;
}

extern "C" bt_status bt_gpt2_create(const bt_gpt2_config* cfg, void* workspace, size_t ws_bytes, int max_B,
                                    int max_T, void* stream, bt_gpt2_ctx** out) {
  bt::clear_error();
  BT_TRY(check_config(cfg));
  BT_RETURN_IF(!out, BT_EINVAL, "bt_gpt2_create: out is NULL");
  BT_RETURN_IF(max_B < 1 || max_T < 1 || max_T > cfg->max_T, BT_ESHAPE,
               "bt_gpt2_create: max_B=%d max_T=%d (cfg max_T=%d)", max_B, max_T, cfg->max_T);
  BT_RETURN_IF((long long)max_B * max_T > (1LL << 26), BT_ESHAPE, "bt_gpt2_create: too many tokens");
  const Layout lay = make_layout(*cfg, max_B, max_T);
  BT_RETURN_IF(!workspace || ws_bytes < lay.total, BT_EWORKSPACE,
               "bt_gpt2_create: workspace of %zu bytes needed (got %zu)", lay.total, ws_bytes);
  BT_RETURN_IF((reinterpret_cast<uintptr_t>(workspace) & 255) != 0, BT_EALIGN,
               "bt_gpt2_create: workspace must be 256-byte aligned");
  bt_gpt2_ctx* c = new bt_gpt2_ctx();
  c->cfg = *cfg;
  c->ws = static_cast<char*>(workspace);
  c->ws_bytes = ws_bytes;
  c->max_B = max_B;
  c->max_T = max_T;
  c->stream = as_stream(stream);
  c->t = 0;
  c->po = param_offsets(*cfg);
  c->lay = lay;
  *out = c;
  return BT_OK;
}

extern "C" void bt_gpt2_destroy(bt_gpt2_ctx* ctx) {
  if (!ctx) return;
  if (!ctx->prof.pool.empty()) {
    (void)hipStreamSynchronize(ctx->stream);
    for (auto& e : ctx->prof.pool) (void)hipEventDestroy(e);
  }
  if (ctx->side) {
    (void)hipStreamSynchronize(ctx->side);
    (void)hipStreamDestroy(ctx->side);
  }
  if (ctx->ev_fork) (void)hipEventDestroy(ctx->ev_fork);
  if (ctx->ev_index) (void)hipEventDestroy(ctx->ev_index);
  delete ctx;
}

extern "C" int bt_gpt2_step_count(const bt_gpt2_ctx* ctx) { return ctx ? ctx->t : -1; }

extern "C" void bt_gpt2_set_step_count(bt_gpt2_ctx* ctx, int t) {
  if (ctx) ctx->t = t;
}

extern "C" bt_status bt_gpt2_read_scalars(const bt_gpt2_ctx* ctx, float* out) {
  bt::clear_error();
  BT_RETURN_IF(!ctx || !out, BT_EINVAL, "bt_gpt2_read_scalars: NULL pointer");
  BT_CHECK_HIP(hipMemcpyAsync(out, ctx->ws + ctx->lay.scalars, 3 * sizeof(float), hipMemcpyDeviceToHost,
                              ctx->stream));
  BT_CHECK_HIP(hipStreamSynchronize(ctx->stream));
  return BT_OK;
}

namespace {

struct StepBufs {
  const bt_gpt2_ctx* c;
  float* f(size_t off) const { return reinterpret_cast<float*>(c->ws + off); }
  float* layer(size_t base, int l) const { return f(base + (size_t)l * c->lay.per_layer); }
  // residual stream input of layer l (l = L is the final residual)
  float* res(int l) const { return l == c->cfg.L ? f(c->lay.resL) : layer(c->lay.res, l); }
  void* scratch() const { return c->ws + c->lay.scratch; }
  size_t scratch_bytes() const { return c->lay.scratch_bytes; }
};

}  // namespace

extern "C" bt_status bt_gpt2_fwd_bwd(bt_gpt2_ctx* ctx, const float* params, float* grads, const int32_t* tokens,
                                     const int32_t* targets, int B, int T, float loss_scale, int accumulate,
                                     float* d_loss, float* loss_rows_out) {
  bt::clear_error();
  BT_RETURN_IF(!ctx || !params || !grads || !tokens || !targets, BT_EINVAL, "bt_gpt2_fwd_bwd: NULL pointer");
  BT_RETURN_IF(B < 1 || T < 1 || B > ctx->max_B || T > ctx->max_T || (long long)B * T > (long long)ctx->max_B * ctx->max_T,
               BT_ESHAPE, "bt_gpt2_fwd_bwd: B=%d T=%d exceed the context's max_B=%d max_T=%d", B, T, ctx->max_B,
               ctx->max_T);
  BT_RETURN_IF(!aligned16(params) || !aligned16(grads), BT_EALIGN, "bt_gpt2_fwd_bwd: params/grads must be 16-byte aligned");
  BT_RETURN_IF(((long long)B * T) % 4 != 0, BT_ESHAPE, "bt_gpt2_fwd_bwd: B*T=%lld must be a multiple of 4",
               (long long)B * T);
  const bt_gpt2_config& cf = ctx->cfg;
  const ParamOffs& po = ctx->po;
  const Layout& ly = ctx->lay;
  prof_break(ctx);  // the caller may have enqueued work since the last call
  StepBufs sb{ctx};
  hipStream_t s = ctx->stream;
  const int M = B * T, C = cf.C, F = 4 * cf.C, H = cf.H, hd = C / H, L = cf.L, Vp = cf.Vp;
  const float beta = accumulate ? 1.f : 0.f;
  const float* P = params;
  float* G = grads;
  void* scr = sb.scratch();
  const size_t scrb = sb.scratch_bytes();
  float* d_scal = sb.f(ly.scalars);
  float* loss_dst = d_loss ? d_loss : d_scal;

  // algorithmic work of each call (FLOPs; bytes with every operand touched once)
  const double fM = M, fC = C, fF = F, fV = Vp, f4 = 4.0;
  auto gemm_f = [](double m, double n, double k) { return 2.0 * m * n * k; };
  auto gemm_b = [&](double m, double n, double k, int extra_mn) { return f4 * (m * k + k * n + (1 + extra_mn) * m * n); };
  const double pairs = (double)B * H * ((double)T * (T + 1) / 2.0);
  const double attn_fwd_f = 4.0 * hd * pairs, attn_bwd_f = 8.0 * hd * pairs;
  const double attn_fwd_b = f4 * (3 * fM * fC + fM * fC + (double)B * H * T);
  const double attn_bwd_b = f4 * (3 * fM * fC + 2 * fM * fC + (double)B * H * T + 3 * fM * fC);
  const double ln_fwd_b = f4 * (2 * fM * fC + 2 * fM + 2 * fC);
  const double ln_bwd_b1 = f4 * (4 * fM * fC + 2 * fM + 3 * fC);  // dx accumulated (read + write)
  const double ln_bwd_b0 = f4 * (3 * fM * fC + 2 * fM + 3 * fC);

  // ---------------- forward
  // token index of the embedding backward, on the side stream (created at
  // the first step): it waits for everything enqueued so far on the main
  // stream (the tokens, and any earlier step still reading the index)
  if (!ctx->side) {
    BT_CHECK_HIP(hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking));
    BT_CHECK_HIP(hipEventCreateWithFlags(&ctx->ev_fork, hipEventDisableTiming));
    BT_CHECK_HIP(hipEventCreateWithFlags(&ctx->ev_index, hipEventDisableTiming));
  }
  void* emb_index = ctx->ws + ly.emb_index;
  const size_t emb_index_b = emb_index_bytes((long long)M);
  BT_CHECK_HIP(hipEventRecord(ctx->ev_fork, s));
  BT_CHECK_HIP(hipStreamWaitEvent(ctx->side, ctx->ev_fork, 0));
  BT_TRY(bt_embedding_index(tokens, emb_index, emb_index_b, B, T, Vp, ctx->side));
  BT_CHECK_HIP(hipEventRecord(ctx->ev_index, ctx->side));
  // every position reads its wte row, wpe rows once per position t, x0 written
  BT_PROF(BT_PROF_EMB_FWD, 0, f4 * (2 * fM * fC + (double)T * fC) + 4.0 * fM,
          bt_embedding_fwd(tokens, P + po.wte, P + po.wpe, sb.res(0), B, T, C, Vp, s));
  for (int l = 0; l < L; ++l) {
    const LayerOffs& w = po.layer[l];
    float* ln1 = sb.layer(ly.ln1, l);
    float* qkv = sb.layer(ly.qkv, l);
    float* att = sb.layer(ly.att, l);
    float* xmid = sb.layer(ly.xmid, l);
    float* ln2 = sb.layer(ly.ln2, l);
    float* hpre = sb.layer(ly.h, l);
    float* gact = sb.layer(ly.g, l);
    BT_PROF(BT_PROF_LN_FWD, 0, ln_fwd_b, bt_layernorm_fwd(sb.res(l), P + w.ln1g, P + w.ln1b, ln1, sb.layer(ly.mu1, l), sb.layer(ly.rs1, l), M, C,
                            cf.ln_eps, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, 3 * fC, fC), gemm_b(fM, 3 * fC, fC, 0), bt_gemm(BT_OP_N, BT_OP_N, M, 3 * C, C, ln1, C, P + w.Wqkv, 3 * C, 0.f, qkv, 3 * C, P + w.bqkv,
                   BT_EPI_BIAS, nullptr, nullptr, nullptr, nullptr, scr, scrb, s));
    BT_PROF(BT_PROF_ATTN_FWD, attn_fwd_f, attn_fwd_b, bt_attention_fwd(qkv, att, sb.layer(ly.lse, l), B, T, H, hd, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fC, fC), gemm_b(fM, fC, fC, 1), bt_gemm(BT_OP_N, BT_OP_N, M, C, C, att, C, P + w.Wo, C, 0.f, xmid, C, P + w.bo, BT_EPI_BIAS, nullptr,
                   nullptr, sb.res(l), nullptr, scr, scrb, s));
    BT_PROF(BT_PROF_LN_FWD, 0, ln_fwd_b, bt_layernorm_fwd(xmid, P + w.ln2g, P + w.ln2b, ln2, sb.layer(ly.mu2, l), sb.layer(ly.rs2, l), M, C,
                            cf.ln_eps, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fF, fC), gemm_b(fM, fF, fC, 1), bt_gemm(BT_OP_N, BT_OP_N, M, F, C, ln2, C, P + w.Wfc, F, 0.f, gact, F, P + w.bfc, BT_EPI_BIAS_GELU, hpre,
                   nullptr, nullptr, nullptr, scr, scrb, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fC, fF), gemm_b(fM, fC, fF, 1), bt_gemm(BT_OP_N, BT_OP_N, M, C, F, gact, F, P + w.Wfp, C, 0.f, sb.res(l + 1), C, P + w.bfp, BT_EPI_BIAS,
                   nullptr, nullptr, xmid, nullptr, scr, scrb, s));
  }
  float* lnf = sb.f(ly.lnf);
  float* logits = sb.f(ly.logits);
  float* lrows = sb.f(ly.loss_rows);
  BT_PROF(BT_PROF_LN_FWD, 0, ln_fwd_b, bt_layernorm_fwd(sb.res(L), P + po.lnfg, P + po.lnfb, lnf, sb.f(ly.muf), sb.f(ly.rsf), M, C, cf.ln_eps, s));
  BT_PROF(BT_PROF_GEMM, gemm_f(fM, fV, fC), gemm_b(fM, fV, fC, 0), bt_gemm(BT_OP_N, BT_OP_T, M, Vp, C, lnf, C, P + po.wte, C, 0.f, logits, Vp, nullptr, BT_EPI_NONE, nullptr,
                 nullptr, nullptr, nullptr, scr, scrb, s));
  // loss rows + dlogits = (softmax - onehot) * loss_scale, written over the logits
  BT_PROF(BT_PROF_XENT, 0, f4 * (2 * fM * fV + 3 * fM), bt_softmax_xent_fused(logits, targets, lrows, sb.f(ly.lse_rows), loss_scale, M, cf.V, Vp, s));
  BT_PROF(BT_PROF_OTHER, 0, f4 * fM, launch_loss_sum(lrows, M, loss_scale, accumulate, loss_dst, s));
  if (loss_rows_out) {
    prof_break(ctx);
    BT_CHECK_HIP(hipMemcpyAsync(loss_rows_out, lrows, sizeof(float) * M, hipMemcpyDeviceToDevice, s));
  }

  // ---------------- backward
  float* dres = sb.f(ly.dres);
  float* dbig = sb.f(ly.dbig);
  float* dsm = sb.f(ly.dsmall);
  const float* dlogits = logits;
  BT_PROF(BT_PROF_GEMM, gemm_f(fM, fC, fV), gemm_b(fM, fC, fV, 0), bt_gemm(BT_OP_N, BT_OP_N, M, C, Vp, dlogits, Vp, P + po.wte, C, 0.f, dsm, C, nullptr, BT_EPI_NONE, nullptr,
                 nullptr, nullptr, nullptr, scr, scrb, s));  // dlnf
  BT_PROF(BT_PROF_GEMM, gemm_f(fV, fC, fM), gemm_b(fV, fC, fM, accumulate), bt_gemm(BT_OP_T, BT_OP_N, Vp, C, M, dlogits, Vp, lnf, C, beta, G + po.wte, C, nullptr, BT_EPI_NONE, nullptr,
                 nullptr, nullptr, nullptr, scr, scrb, s));  // dwte (LM head part)
  // LayerNorm backward: dx now, the dgamma / dbeta partial rows of all 2L+1
  // LayerNorms into their own slabs, summed by one batched launch after the
  // last of them (each sum in the fixed order of bt_layernorm_bwd's)
  std::vector<PartialSet> ln_sets;
  ln_sets.reserve(2 * L + 1);
  auto ln_bwd = [&](const float* dy, const float* x, const float* gam, const float* mu, const float* rs, float dx_beta,
                    float* dgam, float* dbet) {
    float* part = sb.f(ly.ln_part) + ln_sets.size() * ly.ln_part_slab;
    ln_sets.push_back(PartialSet{part, dgam, dbet});
    return ln_bwd_rows(dy, x, gam, mu, rs, dres, dx_beta, part, M, C, s);
  };
  BT_PROF(BT_PROF_LN_BWD, 0, ln_bwd_b0, ln_bwd(dsm, sb.res(L), P + po.lnfg, sb.f(ly.muf), sb.f(ly.rsf), 0.f, G + po.lnfg, G + po.lnfb));
  for (int l = L - 1; l >= 0; --l) {
    const LayerOffs& w = po.layer[l];
    float* ln1 = sb.layer(ly.ln1, l);
    float* qkv = sb.layer(ly.qkv, l);
    float* att = sb.layer(ly.att, l);
    float* xmid = sb.layer(ly.xmid, l);
    float* ln2 = sb.layer(ly.ln2, l);
    float* hpre = sb.layer(ly.h, l);
    float* gact = sb.layer(ly.g, l);
    // MLP down-projection: dWfp += g^T dres and dbfp += colsum(dres) in one product;
    // dh = (dres Wfp^T) * gelu'(h)
    BT_PROF(BT_PROF_GEMM, gemm_f(fF, fC, fM), gemm_b(fF, fC, fM, accumulate), bt_gemm(BT_OP_T, BT_OP_N, F, C, M, gact, F, dres, C, beta, G + w.Wfp, C, nullptr, BT_EPI_NONE, nullptr,
                   nullptr, nullptr, G + w.bfp, scr, scrb, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fF, fC), gemm_b(fM, fF, fC, 1), bt_gemm(BT_OP_N, BT_OP_T, M, F, C, dres, C, P + w.Wfp, C, 0.f, dbig, F, nullptr, BT_EPI_DGELU, nullptr,
                   hpre, nullptr, nullptr, scr, scrb, s));
    // MLP up-projection: dWfc += ln2^T dh with dbfc ; dln2 = dh Wfc^T
    BT_PROF(BT_PROF_GEMM, gemm_f(fC, fF, fM), gemm_b(fC, fF, fM, accumulate), bt_gemm(BT_OP_T, BT_OP_N, C, F, M, ln2, C, dbig, F, beta, G + w.Wfc, F, nullptr, BT_EPI_NONE, nullptr,
                   nullptr, nullptr, G + w.bfc, scr, scrb, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fC, fF), gemm_b(fM, fC, fF, 0), bt_gemm(BT_OP_N, BT_OP_T, M, C, F, dbig, F, P + w.Wfc, F, 0.f, dsm, C, nullptr, BT_EPI_NONE, nullptr,
                   nullptr, nullptr, nullptr, scr, scrb, s));
    BT_PROF(BT_PROF_LN_BWD, 0, ln_bwd_b1, ln_bwd(dsm, xmid, P + w.ln2g, sb.layer(ly.mu2, l), sb.layer(ly.rs2, l), 1.f, G + w.ln2g, G + w.ln2b));
    // attention output projection: dWo += att^T dres with dbo ; datt = dres Wo^T
    BT_PROF(BT_PROF_GEMM, gemm_f(fC, fC, fM), gemm_b(fC, fC, fM, accumulate), bt_gemm(BT_OP_T, BT_OP_N, C, C, M, att, C, dres, C, beta, G + w.Wo, C, nullptr, BT_EPI_NONE, nullptr,
                   nullptr, nullptr, G + w.bo, scr, scrb, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fC, fC), gemm_b(fM, fC, fC, 0), bt_gemm(BT_OP_N, BT_OP_T, M, C, C, dres, C, P + w.Wo, C, 0.f, dsm, C, nullptr, BT_EPI_NONE, nullptr,
                   nullptr, nullptr, nullptr, scr, scrb, s));
    BT_PROF(BT_PROF_ATTN_BWD, attn_bwd_f, attn_bwd_b, bt_attention_bwd(dsm, qkv, att, sb.layer(ly.lse, l), dbig, scr, scrb, B, T, H, hd, s));
    // QKV projection: dWqkv += ln1^T dqkv with dbqkv ; dln1 = dqkv Wqkv^T
    BT_PROF(BT_PROF_GEMM, gemm_f(fC, 3 * fC, fM), gemm_b(fC, 3 * fC, fM, accumulate), bt_gemm(BT_OP_T, BT_OP_N, C, 3 * C, M, ln1, C, dbig, 3 * C, beta, G + w.Wqkv, 3 * C, nullptr, BT_EPI_NONE,
                   nullptr, nullptr, nullptr, G + w.bqkv, scr, scrb, s));
    BT_PROF(BT_PROF_GEMM, gemm_f(fM, fC, 3 * fC), gemm_b(fM, fC, 3 * fC, 0), bt_gemm(BT_OP_N, BT_OP_T, M, C, 3 * C, dbig, 3 * C, P + w.Wqkv, 3 * C, 0.f, dsm, C, nullptr, BT_EPI_NONE,
                   nullptr, nullptr, nullptr, nullptr, scr, scrb, s));
    BT_PROF(BT_PROF_LN_BWD, 0, ln_bwd_b1, ln_bwd(dsm, sb.res(l), P + w.ln1g, sb.layer(ly.mu1, l), sb.layer(ly.rs1, l), 1.f, G + w.ln1g, G + w.ln1b));
  }
  BT_PROF(BT_PROF_LN_BWD, 0, 0, sum_partials_batched(ln_sets.data(), (int)ln_sets.size(), ln_bwd_partial_rows(M, C), 2LL * C, 2 * C, C, beta, s));
  // dx0 read once, dwpe written (and read when accumulating); the dwte rows of
  // the distinct tokens (read + written) depend on the data and are not counted here
  prof_break(ctx);
  BT_CHECK_HIP(hipStreamWaitEvent(s, ctx->ev_index, 0));
  BT_PROF(BT_PROF_EMB_BWD, 0, f4 * (fM * fC + (1.0 + beta) * (double)T * fC),
          bt_embedding_bwd_indexed(emb_index, emb_index_b, dres, G + po.wte, G + po.wpe, beta, scr, scrb, B, T, C, Vp, s));
  // rows of wpe beyond T receive no gradient in this micro-step
  if (T < cf.max_T && !accumulate) {
    prof_break(ctx);
    BT_TRY(fill_zero(G + po.wpe + (size_t)T * C, (size_t)(cf.max_T - T) * C, s));
  }
  return BT_OK;
}

extern "C" bt_status bt_gpt2_optimizer_step(bt_gpt2_ctx* ctx, float* params, float* grads, float* opt_state, int t,
                                            double lr) {
  bt::clear_error();
  BT_RETURN_IF(!ctx || !params || !grads || !opt_state, BT_EINVAL, "bt_gpt2_optimizer_step: NULL pointer");
  BT_RETURN_IF(t < 1, BT_EINVAL, "bt_gpt2_optimizer_step: t=%d must be >= 1", t);
  const bt_gpt2_config& cf = ctx->cfg;
  const size_t P = ctx->po.total;
  prof_break(ctx);
  StepBufs sb{ctx};
  float* d_scal = sb.f(ctx->lay.scalars);
  // the coefficient is 1 without clipping and NaN when the norm is not
  // finite, in which case the AdamW launch writes nothing
  BT_PROF(BT_PROF_GRAD_NORM, 2.0 * P, 4.0 * P,
          bt_grad_norm_clip(grads, P, (float)cf.grad_clip, d_scal + 1, d_scal + 2, sb.scratch(), sb.scratch_bytes(),
                            ctx->stream));
  BT_PROF(BT_PROF_ADAMW, 0, 28.0 * P,
          bt_adamw_step(params, grads, opt_state, opt_state + P, P, ctx->po.n_decay, lr, cf.beta1, cf.beta2,
                        cf.adam_eps, cf.weight_decay, t, d_scal + 2, ctx->stream));
  return BT_OK;
}

extern "C" float bt_gpt2_train_step(bt_gpt2_ctx* ctx, float* params, float* grads, float* opt_state,
                                    const int32_t* tokens, const int32_t* targets, int B, int T) {
  bt::clear_error();
  if (!ctx) {
    fail(BT_EINVAL, "bt_gpt2_train_step: ctx is NULL");
    return NAN;
  }
  StepBufs sb{ctx};
  float* d_scal = sb.f(ctx->lay.scalars);  // [loss, norm, coef]
  const float scale = 1.0f / (float)((double)B * T);
  if (bt_gpt2_fwd_bwd(ctx, params, grads, tokens, targets, B, T, scale, 0, d_scal, nullptr) != BT_OK) return NAN;
  if (bt_gpt2_optimizer_step(ctx, params, grads, opt_state, ctx->t + 1, ctx->cfg.lr) != BT_OK) return NAN;
  float h[3] = {NAN, NAN, NAN};
  hipError_t e = hipMemcpyAsync(h, d_scal, sizeof(h), hipMemcpyDeviceToHost, ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) {
    fail(BT_EHIP, "bt_gpt2_train_step: %s", hipGetErrorString(e));
    return NAN;
  }
  if (ctx->prof.on && prof_flush(ctx) != BT_OK) return NAN;
  if (!std::isfinite(h[1])) {
    // AdamW wrote nothing; the step counter stays
    fail(BT_ENONFINITE, "bt_gpt2_train_step: non-finite gradient norm (%g, loss %g); parameters and moments "
                        "not updated", (double)h[1], (double)h[0]);
    return NAN;
  }
  ctx->t += 1;
  return h[0];
}
