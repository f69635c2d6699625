// graft_api.hip -- host side of the C ABI declared in include/graft.h:
// validation, context and workspace ownership, kernel launches on the
// caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>

#include "graft_internal.h"

// The per-round intermediates of graft_build_tree_static live here instead of
// in a context's workspace: one copy per GPU, held until the process ends.
// Host code never uses this name as an address; it resolves the device address
// once per device with hipGetSymbolAddress (static_scratch_on) and passes that.
static __device__ __align__(256) uint64_t scratch[GRAFT_STATIC_SCRATCH_BYTES / 8];

namespace graft {

int64_t carve_round_scratch(const graft_dims &d, int batch, int64_t part_slots, char *base,
                            RoundScratch *ws) {
  const int64_t B = batch, L = d.num_pos, K = d.top_k;
  int64_t off = 0;
  auto take = [&](int64_t bytes) -> char * {
    char *p = base ? base + off : nullptr;
    off += (bytes + 255) & ~int64_t{255};
    return p;
  };
  RoundScratch w{};
  w.part_slots = part_slots;
  w.part_stats = reinterpret_cast<double *>(take(part_slots * 3 * int64_t{sizeof(double)}));
  w.part_keys = reinterpret_cast<uint64_t *>(take(part_slots * K * int64_t{sizeof(uint64_t)}));
  w.topk_ids = reinterpret_cast<int32_t *>(take(B * L * K * int64_t{sizeof(int32_t)}));
  w.topk_logq = reinterpret_cast<float *>(take(B * L * K * int64_t{sizeof(float)}));
  w.row_stats = reinterpret_cast<float *>(take(B * L * 3 * int64_t{sizeof(float)}));
  w.edge_rows = reinterpret_cast<float *>(take(B * L * K * K * int64_t{sizeof(float)}));
  w.cand_by_rank = reinterpret_cast<int32_t *>(take(B * L * K * int64_t{sizeof(int32_t)}));
  w.positive = reinterpret_cast<uint8_t *>(take(B * L));
  w.adj_cos = reinterpret_cast<float *>(take(B * (L > 1 ? L - 1 : 1) * int64_t{sizeof(float)}));
  if (ws) *ws = w;
  return off;
}

}  // namespace graft

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device dev, which must be current: resolved
// on first use per device and kept for the life of the process.
hipError_t static_scratch_on(int dev, char **out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = static_cast<char *>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char *what) {
  return fail(GRAFT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

template <typename T>
hipError_t dalloc(T **p, size_t n) {
  *p = nullptr;
  if (n == 0) n = 1;
  return hipMalloc(reinterpret_cast<void **>(p), n * sizeof(T));
}

void prof_release(graft_ctx *c) {
  if (c->prof_build) {
    for (int i = 0; i < 4 * c->prof_cap; ++i) (void)hipEventDestroy(c->prof_build[i]);
    for (int i = 0; i < 2 * c->prof_cap; ++i) (void)hipEventDestroy(c->prof_acc[i]);
    delete[] c->prof_build;
    delete[] c->prof_acc;
  }
  c->prof_build = c->prof_acc = nullptr;
  c->prof_cap = c->prof_nbuild = c->prof_nacc = 0;
}

void free_ctx(graft_ctx *c) {
  if (!c) return;
  prof_release(c);
  (void)hipFree(c->ws_base);
  (void)hipFree(c->proj_parent);
  (void)hipFree(c->proj_child);
  (void)hipFree(c->depth_emb);
  (void)hipFree(c->hist_ring);
  (void)hipFree(c->hist_pos);
  (void)hipFree(c->error_flag);
  delete c;
}

// Steps 1-5 of a round (graft_build_tree, graft_build_tree_static) with the
// per-round intermediates in ws; `who` names the entry point in messages.
int build_tree_with(graft_ctx *ctx, const graft_round_in *in, const graft_tree_out *out,
                    const graft::RoundScratch &ws, graft_stream_t stream, const char *who) {
  if (!ctx || !in || !out) return fail(GRAFT_ERR_INVALID_ARG, "%s: NULL argument", who);
  const graft_dims &d = ctx->dims;
  if (in->batch < 1 || in->batch > d.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "%s: batch %d outside 1..%d", who, in->batch,
                d.max_batch);
  if (!in->logits || !in->root_token || !in->base_pos)
    return fail(GRAFT_ERR_INVALID_ARG, "%s: logits, root_token and base_pos are required", who);
  if ((reinterpret_cast<uintptr_t>(in->logits) & 15u) != 0)
    return fail(GRAFT_ERR_INVALID_ARG, "%s: logits must be 16-byte aligned", who);
  if (!out->budget || !out->n_nodes || !out->tokens || !out->parents || !out->pos_ids)
    return fail(GRAFT_ERR_INVALID_ARG,
                "%s: budget, n_nodes, tokens, parents and pos_ids are required", who);
  if (!ctx->has_scorer)
    return fail(GRAFT_ERR_INVALID_ARG, "%s: no scorer installed (graft_set_scorer)", who);
  if (!in->fixed_budget && !ctx->has_saba)
    return fail(GRAFT_ERR_INVALID_ARG,
                "%s: no fixed budgets and no SABA parameters (graft_set_saba)", who);
  if (in->hidden) {
    if (in->hidden_dim < 8 || in->hidden_dim > (1 << 20) || (in->hidden_dim & 7) != 0)
      return fail(GRAFT_ERR_INVALID_ARG, "%s: hidden_dim %d must be a multiple of 8 in 8..1048576",
                  who, in->hidden_dim);
    if ((reinterpret_cast<uintptr_t>(in->hidden) & 15u) != 0)
      return fail(GRAFT_ERR_INVALID_ARG, "%s: hidden must be 16-byte aligned", who);
  }
  if (!in->hist && !in->fixed_budget && !ctx->has_history)
    return fail(GRAFT_ERR_INVALID_ARG,
                "%s: no hist input and no history ring (graft_set_history)", who);
  char what[96];
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipEvent_t *ev = nullptr;
  if (ctx->prof_build && ctx->prof_nbuild < ctx->prof_cap) ev = ctx->prof_build + 4 * ctx->prof_nbuild++;
  if (ev) (void)hipEventRecord(ev[0], s);
  hipError_t e = graft::launch_logits_pass(ctx, ws, in->batch, in->logits, out, s);
  if (e != hipSuccess) {
    snprintf(what, sizeof what, "%s: logits pass", who);
    return hip_fail(e, what);
  }
  if (ev) (void)hipEventRecord(ev[1], s);
  if (in->hidden) {
    e = graft::launch_degen(ctx, ws, in->batch, in->hidden, in->hidden_dim, out->adj_cos, s);
    if (e != hipSuccess) {
      snprintf(what, sizeof what, "%s: hidden-state cosines", who);
      return hip_fail(e, what);
    }
  }
  if (!graft::edges_fused(ctx)) e = graft::launch_edge_scores(ctx, ws, in, out, s);
  if (e != hipSuccess) {
    snprintf(what, sizeof what, "%s: edge scores and budget", who);
    return hip_fail(e, what);
  }
  if (ev) (void)hipEventRecord(ev[2], s);
  e = graft::launch_select(ctx, ws, in, out, s);
  if (e != hipSuccess) {
    snprintf(what, sizeof what, "%s: selection", who);
    return hip_fail(e, what);
  }
  if (ev) (void)hipEventRecord(ev[3], s);
  return GRAFT_OK;
}

}  // namespace

extern "C" {

const char *graft_status_string(int s) {
  switch (s) {
    case GRAFT_OK: return "ok";
    case GRAFT_ERR_INVALID_ARG: return "invalid argument";
    case GRAFT_ERR_UNSUPPORTED: return "unsupported size";
    case GRAFT_ERR_OUT_OF_MEMORY: return "out of device memory";
    case GRAFT_ERR_HIP: return "HIP runtime error";
    case GRAFT_ERR_DEVICE_DATA: return "invalid data seen on the device";
    default: return "unknown status";
  }
}

const char *graft_last_error(void) { return g_err; }

int graft_create(const graft_dims *dims, graft_ctx **out) {
  if (!dims || !out) return fail(GRAFT_ERR_INVALID_ARG, "graft_create: NULL argument");
  *out = nullptr;
  graft_dims d = *dims;
  if (d.hist_window == 0) d.hist_window = 4;
  if (d.max_batch < 1 || d.num_pos < 1 || d.vocab < 1 || d.top_k < 1 || d.max_nodes < 1 ||
      d.hist_window < 1)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_create: sizes must be positive");
  if (d.num_pos > graft::kMaxL)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_create: num_pos %d > %d", d.num_pos, graft::kMaxL);
  if (d.top_k > graft::kMaxK)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_create: top_k %d > %d", d.top_k, graft::kMaxK);
  if (d.top_k > d.vocab)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_create: top_k %d > vocab %d", d.top_k, d.vocab);
  if (d.max_nodes > graft::kMaxNodes)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_create: max_nodes %d > %d", d.max_nodes,
                graft::kMaxNodes);
  if (d.hist_window > 64)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_create: hist_window %d > 64", d.hist_window);
  if (static_cast<int64_t>(d.max_batch) * d.num_pos > (1 << 24))
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_create: max_batch * num_pos too large");

  graft_ctx *c = new (std::nothrow) graft_ctx();
  if (!c) return fail(GRAFT_ERR_OUT_OF_MEMORY, "graft_create: host allocation failed");
  c->dims = d;
  c->fuse_edges = true;
  (void)hipGetDevice(&c->device);
  const size_t B = d.max_batch;
  const int64_t ws_bytes =
      graft::carve_round_scratch(d, d.max_batch, graft::logits_part_slots(d), nullptr, nullptr);
  hipError_t e = dalloc(&c->ws_base, static_cast<size_t>(ws_bytes));
  if (e == hipSuccess)
    graft::carve_round_scratch(d, d.max_batch, graft::logits_part_slots(d), c->ws_base, &c->ws);
  if (e == hipSuccess) e = static_scratch_on(c->device, &c->static_scratch);
#define GRAFT_ALLOC(ptr, n)              \
  if (e == hipSuccess) e = dalloc(&(ptr), (n));
  GRAFT_ALLOC(c->hist_ring, B * d.hist_window);
  GRAFT_ALLOC(c->hist_pos, B);
  GRAFT_ALLOC(c->error_flag, 1);
#undef GRAFT_ALLOC
  if (e == hipSuccess) e = hipMemset(c->error_flag, 0, sizeof(uint32_t));
  if (e == hipSuccess) e = hipMemset(c->hist_ring, 0, B * d.hist_window * sizeof(int32_t));
  if (e == hipSuccess) e = hipMemset(c->hist_pos, 0, B * sizeof(int32_t));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    free_ctx(c);
    return e == hipErrorOutOfMemory ? fail(GRAFT_ERR_OUT_OF_MEMORY, "graft_create: %s",
                                           hipGetErrorString(e))
                                    : hip_fail(e, "graft_create");
  }
  *out = c;
  return GRAFT_OK;
}

void graft_destroy(graft_ctx *ctx) {
  if (!ctx) return;
  (void)hipDeviceSynchronize();
  free_ctx(ctx);
}

int graft_set_fusion(graft_ctx *ctx, int32_t enable, int32_t *active) {
  if (!ctx) return fail(GRAFT_ERR_INVALID_ARG, "graft_set_fusion: NULL context");
  ctx->fuse_edges = enable != 0;
  if (active) *active = ctx->has_scorer && graft::edges_fused(ctx) ? 1 : 0;
  return GRAFT_OK;
}

int graft_set_scorer(graft_ctx *ctx, const graft_scorer_desc *desc, graft_stream_t stream) {
  if (!ctx || !desc) return fail(GRAFT_ERR_INVALID_ARG, "graft_set_scorer: NULL argument");
  if (!desc->emb || !desc->g_parent || !desc->g_child)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_scorer: emb, g_parent and g_child are required");
  if (desc->emb_dim < 1 || desc->score_dim < 1)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_scorer: emb_dim and score_dim must be positive");
  if (desc->score_dim > graft::kMaxScoreDim)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_set_scorer: score_dim %d > %d", desc->score_dim,
                graft::kMaxScoreDim);
  if (!std::isfinite(desc->scale) || !std::isfinite(desc->beta))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_scorer: scale and beta must be finite");
  const size_t V = ctx->dims.vocab, m = desc->score_dim, L = ctx->dims.num_pos;
  hipError_t e = hipSuccess;
  if (ctx->scorer.score_dim != desc->score_dim || !ctx->proj_parent) {
    (void)hipStreamSynchronize(reinterpret_cast<hipStream_t>(stream));
    (void)hipFree(ctx->proj_parent);
    (void)hipFree(ctx->proj_child);
    (void)hipFree(ctx->depth_emb);
    ctx->proj_parent = ctx->proj_child = ctx->depth_emb = nullptr;
    ctx->has_scorer = false;
    e = dalloc(&ctx->proj_parent, V * m);
    if (e == hipSuccess) e = dalloc(&ctx->proj_child, V * m);
    if (e == hipSuccess) e = dalloc(&ctx->depth_emb, L * m);
    if (e != hipSuccess) return hip_fail(e, "graft_set_scorer: allocation");
  }
  ctx->scorer.scale = desc->scale;
  ctx->scorer.beta = desc->beta;
  ctx->scorer.center = desc->center != 0;
  ctx->scorer.score_dim = desc->score_dim;
  ctx->scorer.has_depth_emb = desc->depth_emb != nullptr;
  if (desc->depth_emb) {
    e = hipMemcpyAsync(ctx->depth_emb, desc->depth_emb, L * m * sizeof(float),
                       hipMemcpyDeviceToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "graft_set_scorer: depth embedding copy");
  }
  e = graft::launch_projection(ctx, desc, stream);
  if (e != hipSuccess) return hip_fail(e, "graft_set_scorer: projection launch");
  ctx->has_scorer = true;
  return GRAFT_OK;
}

int graft_set_saba(graft_ctx *ctx, const graft_saba_desc *desc) {
  if (!ctx || !desc || !desc->budgets)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_saba: NULL argument");
  if (desc->n_budgets < 1 || desc->n_budgets > graft::kMaxGrid)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_set_saba: n_budgets must be in 1..%d",
                graft::kMaxGrid);
  for (int i = 0; i < desc->n_budgets; ++i) {
    const int v = desc->budgets[i];
    if (v < 1 || v > ctx->dims.max_nodes)
      return fail(GRAFT_ERR_INVALID_ARG, "graft_set_saba: budget %d outside 1..max_nodes", v);
    if (i > 0 && v <= desc->budgets[i - 1])
      return fail(GRAFT_ERR_INVALID_ARG, "graft_set_saba: budgets must be strictly ascending");
  }
  if (!(desc->tau_min > 0.f) || !std::isfinite(desc->tau_min))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_saba: tau_min must be positive and finite");
  for (int i = 0; i < 4; ++i)
    if (!std::isfinite(desc->phi[i]))
      return fail(GRAFT_ERR_INVALID_ARG, "graft_set_saba: phi must be finite");
  if (!std::isfinite(desc->c0) || !std::isfinite(desc->c1) || !std::isfinite(desc->c2))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_saba: cost coefficients must be finite");
  graft::SabaParams p{};
  for (int i = 0; i < desc->n_budgets; ++i) p.grid[i] = desc->budgets[i];
  p.n_grid = desc->n_budgets;
  for (int i = 0; i < 4; ++i) p.phi[i] = desc->phi[i];
  p.tau_min = desc->tau_min;
  p.c0 = desc->c0;
  p.c1 = desc->c1;
  p.c2 = desc->c2;
  ctx->saba = p;
  ctx->has_saba = true;
  return GRAFT_OK;
}

int graft_set_history(graft_ctx *ctx, int32_t batch, const int32_t *init, graft_stream_t stream) {
  if (!ctx || !init) return fail(GRAFT_ERR_INVALID_ARG, "graft_set_history: NULL argument");
  if (batch < 1 || batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_set_history: batch %d outside 1..%d", batch,
                ctx->dims.max_batch);
  hipError_t e = graft::launch_set_history(ctx, batch, init, stream);
  if (e != hipSuccess) return hip_fail(e, "graft_set_history");
  ctx->has_history = true;
  return GRAFT_OK;
}

int graft_get_history(graft_ctx *ctx, int32_t batch, int32_t *ring, int32_t *pos,
                      graft_stream_t stream) {
  if (!ctx || !ring) return fail(GRAFT_ERR_INVALID_ARG, "graft_get_history: NULL argument");
  if (batch < 1 || batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_get_history: batch %d outside 1..%d", batch,
                ctx->dims.max_batch);
  if (!ctx->has_history)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_get_history: no history ring (graft_set_history)");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(ring, ctx->hist_ring,
                                sizeof(int32_t) * batch * ctx->dims.hist_window,
                                hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess && pos)
    e = hipMemcpyAsync(pos, ctx->hist_pos, sizeof(int32_t) * batch, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "graft_get_history");
  return GRAFT_OK;
}

int graft_build_tree(graft_ctx *ctx, const graft_round_in *in, const graft_tree_out *out,
                     graft_stream_t stream) {
  if (!ctx) return fail(GRAFT_ERR_INVALID_ARG, "graft_build_tree: NULL argument");
  return build_tree_with(ctx, in, out, ctx->ws, stream, "graft_build_tree");
}

int graft_build_tree_static(graft_ctx *ctx, const graft_round_in *in, const graft_tree_out *out,
                            graft_stream_t stream) {
  if (!ctx || !in || !out)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_build_tree_static: NULL argument");
  if (in->batch < 1 || in->batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_build_tree_static: batch %d outside 1..%d",
                in->batch, ctx->dims.max_batch);
  if (!ctx->static_scratch)
    return fail(GRAFT_ERR_HIP, "graft_build_tree_static: no static scratch on device %d",
                ctx->device);
  const int rows = in->batch * ctx->dims.num_pos;
  const int splits = graft::logits_splits(ctx->dims, rows);
  const int64_t parts = splits > 1 ? static_cast<int64_t>(rows) * splits : 0;
  const int64_t need = graft::carve_round_scratch(ctx->dims, in->batch, parts, nullptr, nullptr);
  if (need > GRAFT_STATIC_SCRATCH_BYTES)
    return fail(GRAFT_ERR_UNSUPPORTED,
                "graft_build_tree_static: a batch of %d needs %lld bytes of scratch; the static "
                "buffer holds %lld (use graft_build_tree or a smaller batch)",
                in->batch, static_cast<long long>(need),
                static_cast<long long>(GRAFT_STATIC_SCRATCH_BYTES));
  graft::RoundScratch ws;
  graft::carve_round_scratch(ctx->dims, in->batch, parts, ctx->static_scratch, &ws);
  return build_tree_with(ctx, in, out, ws, stream, "graft_build_tree_static");
}

int graft_accept(graft_ctx *ctx, int32_t batch, const int32_t *n_nodes, const int32_t *tokens,
                 const int32_t *parents, const graft_targets *targets, int32_t *acc_len,
                 int32_t *acc_nodes, int32_t *bonus, int32_t update_history,
                 graft_stream_t stream) {
  if (!ctx || !targets || !n_nodes || !tokens || !parents || !acc_len || !acc_nodes || !bonus)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_accept: NULL argument");
  if (batch < 1 || batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_accept: batch %d outside 1..%d", batch,
                ctx->dims.max_batch);
  const bool per_node = targets->target_node != nullptr;
  const bool per_depth = targets->target_depth != nullptr;
  if (per_node == per_depth)
    return fail(GRAFT_ERR_INVALID_ARG,
                "graft_accept: give exactly one of target_node and target_depth");
  if (per_node && !targets->target_root)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_accept: per-node targets need target_root");
  if (update_history && !ctx->has_history)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_accept: no history ring (graft_set_history)");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipEvent_t *ev = nullptr;
  if (ctx->prof_acc && ctx->prof_nacc < ctx->prof_cap) ev = ctx->prof_acc + 2 * ctx->prof_nacc++;
  if (ev) (void)hipEventRecord(ev[0], s);
  hipError_t e = graft::launch_accept(ctx, batch, n_nodes, tokens, parents, targets, acc_len,
                                      acc_nodes, bonus, update_history, s);
  if (e != hipSuccess) return hip_fail(e, "graft_accept");
  if (ev) (void)hipEventRecord(ev[1], s);
  return GRAFT_OK;
}

int graft_mask_to_bias(graft_ctx *ctx, int32_t batch, const int32_t *n_nodes,
                       const uint64_t *mask, void *bias, int32_t dtype, int64_t ld,
                       int64_t batch_stride, graft_stream_t stream) {
  if (!ctx || !n_nodes || !mask || !bias)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_mask_to_bias: NULL argument");
  if (batch < 1 || batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_mask_to_bias: batch %d outside 1..%d", batch,
                ctx->dims.max_batch);
  if (dtype != 0 && dtype != 1)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_mask_to_bias: dtype %d is neither 0 (fp32) nor 1 (bf16)",
                dtype);
  const int64_t n_max = ctx->dims.max_nodes, per = dtype == 1 ? 8 : 4;
  if (ld < n_max || (batch > 1 && batch_stride < n_max * ld))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_mask_to_bias: ld or batch_stride too small");
  if ((reinterpret_cast<uintptr_t>(bias) & 15u) != 0 || ld % per != 0 || batch_stride % per != 0)
    return fail(GRAFT_ERR_INVALID_ARG,
                "graft_mask_to_bias: bias must be 16-byte aligned with ld and batch_stride "
                "multiples of %d elements", static_cast<int>(per));
  hipError_t e = graft::launch_mask_to_bias(ctx, batch, n_nodes, mask, bias, dtype, ld,
                                            batch_stride, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "graft_mask_to_bias");
  return GRAFT_OK;
}

int graft_commit_accepted(graft_ctx *ctx, int32_t batch, const int32_t *acc_len,
                          const int32_t *acc_nodes, const void *src, void *dst, int64_t row_bytes,
                          int32_t n_planes, int64_t src_plane_stride, int64_t src_batch_stride,
                          int64_t src_row_stride, int64_t dst_plane_stride,
                          int64_t dst_batch_stride, int64_t dst_row_stride,
                          graft_stream_t stream) {
  if (!ctx || !acc_len || !acc_nodes || !src || !dst)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_commit_accepted: NULL argument");
  if (batch < 1 || batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_commit_accepted: batch %d outside 1..%d", batch,
                ctx->dims.max_batch);
  if (n_planes < 1 || row_bytes < 16)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_commit_accepted: need n_planes >= 1, row_bytes >= 16");
  const int64_t v[7] = {row_bytes, src_plane_stride, src_batch_stride, src_row_stride,
                        dst_plane_stride, dst_batch_stride, dst_row_stride};
  for (int i = 0; i < 7; ++i)
    if (v[i] < 0 || v[i] % 16 != 0)
      return fail(GRAFT_ERR_INVALID_ARG,
                  "graft_commit_accepted: row_bytes and strides must be non-negative multiples of 16");
  if (((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u) != 0)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_commit_accepted: src and dst must be 16-byte aligned");
  const int64_t chunks = (row_bytes + 4095) / 4096;
  if (static_cast<int64_t>(n_planes) * batch * chunks >= (int64_t{1} << 31))
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_commit_accepted: too many rows to move in one call");
  hipError_t e = graft::launch_commit(ctx, batch, acc_len, acc_nodes, src, dst, row_bytes,
                                      n_planes, src_plane_stride, src_batch_stride,
                                      src_row_stride, dst_plane_stride, dst_batch_stride,
                                      dst_row_stride, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "graft_commit_accepted");
  return GRAFT_OK;
}

int graft_get_device_status(graft_ctx *ctx, graft_stream_t stream) {
  if (!ctx) return fail(GRAFT_ERR_INVALID_ARG, "graft_get_device_status: NULL context");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint32_t flag = 0;
  hipError_t e = hipMemcpyAsync(&flag, ctx->error_flag, sizeof flag, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "graft_get_device_status");
  if (flag) {
    e = hipMemsetAsync(ctx->error_flag, 0, sizeof flag, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "graft_get_device_status: clear");
    return fail(GRAFT_ERR_DEVICE_DATA, "kernels saw invalid data (flags 0x%x)", flag);
  }
  return GRAFT_OK;
}

int graft_profile_begin(graft_ctx *ctx, int32_t max_calls) {
  if (!ctx || max_calls < 1 || max_calls > (1 << 20))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_profile_begin: bad arguments");
  prof_release(ctx);
  ctx->prof_build = new (std::nothrow) hipEvent_t[4 * static_cast<size_t>(max_calls)];
  ctx->prof_acc = new (std::nothrow) hipEvent_t[2 * static_cast<size_t>(max_calls)];
  if (!ctx->prof_build || !ctx->prof_acc) {
    delete[] ctx->prof_build;
    delete[] ctx->prof_acc;
    ctx->prof_build = ctx->prof_acc = nullptr;
    return fail(GRAFT_ERR_OUT_OF_MEMORY, "graft_profile_begin: host allocation failed");
  }
  ctx->prof_cap = 0;
  for (int i = 0; i < max_calls; ++i) {
    hipError_t e = hipSuccess;
    // timing-only events: no system-scope fence (cache writeback and
    // invalidation) when they are recorded, which would add to the stages
    for (int j = 0; j < 4 && e == hipSuccess; ++j)
      e = hipEventCreateWithFlags(&ctx->prof_build[4 * i + j], hipEventDisableSystemFence);
    for (int j = 0; j < 2 && e == hipSuccess; ++j)
      e = hipEventCreateWithFlags(&ctx->prof_acc[2 * i + j], hipEventDisableSystemFence);
    if (e != hipSuccess) {
      prof_release(ctx);
      return hip_fail(e, "graft_profile_begin: hipEventCreate");
    }
    ctx->prof_cap = i + 1;
  }
  ctx->prof_nbuild = ctx->prof_nacc = 0;
  return GRAFT_OK;
}

int graft_profile_end(graft_ctx *ctx, double *stage_ms, int32_t *stage_calls) {
  if (!ctx || !stage_ms || !stage_calls)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_profile_end: NULL argument");
  for (int j = 0; j < 4; ++j) {
    stage_ms[j] = 0.0;
    stage_calls[j] = 0;
  }
  if (!ctx->prof_build) return fail(GRAFT_ERR_INVALID_ARG, "graft_profile_end: not armed");
  hipError_t e = hipSuccess;
  for (int i = 0; i < ctx->prof_nbuild && e == hipSuccess; ++i) {
    hipEvent_t *ev = ctx->prof_build + 4 * i;
    e = hipEventSynchronize(ev[3]);
    for (int j = 0; j < 3 && e == hipSuccess; ++j) {
      float ms = 0.f;
      e = hipEventElapsedTime(&ms, ev[j], ev[j + 1]);
      stage_ms[j] += ms;
      stage_calls[j] += 1;
    }
  }
  for (int i = 0; i < ctx->prof_nacc && e == hipSuccess; ++i) {
    hipEvent_t *ev = ctx->prof_acc + 2 * i;
    float ms = 0.f;
    e = hipEventSynchronize(ev[1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev[0], ev[1]);
    stage_ms[3] += ms;
    stage_calls[3] += 1;
  }
  prof_release(ctx);
  if (e != hipSuccess) return hip_fail(e, "graft_profile_end");
  return GRAFT_OK;
}

int graft_synth_node_targets(graft_ctx *ctx, int32_t batch, uint64_t seed,
                             const int32_t *root_token, const int32_t *n_nodes,
                             const int32_t *tokens, const int32_t *parents,
                             const int32_t *topk_ids, int32_t *target_root, int32_t *target_node,
                             graft_stream_t stream) {
  if (!ctx || !root_token || !n_nodes || !tokens || !parents || !topk_ids || !target_root ||
      !target_node)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_synth_node_targets: NULL argument");
  if (batch < 1 || batch > ctx->dims.max_batch)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_synth_node_targets: batch %d outside 1..%d", batch,
                ctx->dims.max_batch);
  hipError_t e = graft::launch_synth_targets(ctx, batch, seed, root_token, n_nodes, tokens,
                                             parents, topk_ids, target_root, target_node,
                                             reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "graft_synth_node_targets");
  return GRAFT_OK;
}

}  // extern "C"

namespace {

// Solves the n x n system M x = r (row-major, n <= 4) by Gaussian elimination
// with partial pivoting; false when a pivot is not positive enough.
bool solve_small(int n, double *M, double *r, double *x) {
  for (int c = 0; c < n; ++c) {
    int p = c;
    for (int i = c + 1; i < n; ++i)
      if (std::fabs(M[i * n + c]) > std::fabs(M[p * n + c])) p = i;
    if (!(std::fabs(M[p * n + c]) > 1e-300)) return false;
    if (p != c) {
      for (int j = 0; j < n; ++j) std::swap(M[c * n + j], M[p * n + j]);
      std::swap(r[c], r[p]);
    }
    for (int i = c + 1; i < n; ++i) {
      const double f = M[i * n + c] / M[c * n + c];
      for (int j = c; j < n; ++j) M[i * n + j] -= f * M[c * n + j];
      r[i] -= f * r[c];
    }
  }
  for (int c = n - 1; c >= 0; --c) {
    double v = r[c];
    for (int j = c + 1; j < n; ++j) v -= M[c * n + j] * x[j];
    x[c] = v / M[c * n + c];
    if (!std::isfinite(x[c])) return false;
  }
  return true;
}

// Symmetric matrix from its upper triangle (row by row).
void unpack_sym(int n, const double *u, double *M) {
  int k = 0;
  for (int p = 0; p < n; ++p)
    for (int q = p; q < n; ++q) M[p * n + q] = M[q * n + p] = u[k++];
}

}  // namespace

extern "C" {

int graft_read_stream(const void *src, int64_t bytes, uint32_t *sink, graft_stream_t stream) {
  if (!src || !sink) return fail(GRAFT_ERR_INVALID_ARG, "graft_read_stream: NULL argument");
  if (bytes <= 0 || (bytes & 15) != 0)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_read_stream: bytes %lld is not a positive multiple of 16",
                static_cast<long long>(bytes));
  if ((reinterpret_cast<uintptr_t>(src) & 15) != 0 || (reinterpret_cast<uintptr_t>(sink) & 3) != 0)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_read_stream: misaligned src or sink");
  hipError_t e = graft::launch_read_stream(src, bytes, sink, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "graft_read_stream");
  return GRAFT_OK;
}

int graft_saba_fit(const graft_saba_replay *log, const float *phi_init, int32_t max_iter,
                   float *phi_out, float *c_out, double *stats, graft_stream_t stream) {
  if (!log || !phi_init || !phi_out || !c_out)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_saba_fit: NULL argument");
  const int T = log->n_rounds, nb = log->n_budgets;
  if (T < 1 || nb < 1 || nb > 64 || max_iter < 0)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_saba_fit: need n_rounds >= 1, n_budgets in 1..64, max_iter >= 0");
  if (!log->budgets || !log->state || !log->prefix || !log->accepted || !log->latency)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_saba_fit: a log array is NULL");
  if (!(log->tau_min > 0.0f) || !std::isfinite(log->tau_min))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_saba_fit: tau_min must be positive and finite");
  for (int j = 0; j < nb; ++j)
    if (log->budgets[j] < 1) return fail(GRAFT_ERR_INVALID_ARG, "graft_saba_fit: budgets must be positive");
  for (int k = 0; k < 4; ++k)
    if (!std::isfinite(phi_init[k])) return fail(GRAFT_ERR_INVALID_ARG, "graft_saba_fit: phi_init must be finite");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int32_t *d_budgets = nullptr;
  double *d_part = nullptr, *d_out = nullptr;
  hipError_t e = dalloc(&d_budgets, static_cast<size_t>(nb));
  if (e == hipSuccess) e = dalloc(&d_part, static_cast<size_t>(graft::kFitMaxBlocks) * graft::kFitSums);
  if (e == hipSuccess) e = dalloc(&d_out, static_cast<size_t>(graft::kFitSums));
  if (e == hipSuccess)
    e = hipMemcpyAsync(d_budgets, log->budgets, sizeof(int32_t) * nb, hipMemcpyHostToDevice, s);
  double sums[graft::kFitSums];
  const double tau_min = log->tau_min;
  auto eval = [&](const double *phi, int with_cost, const double *cfit) -> hipError_t {
    hipError_t err = graft::launch_replay_sums(T, nb, d_budgets, log->state, log->prefix,
                                               log->accepted, log->latency, phi, tau_min, with_cost,
                                               cfit, d_part, d_out, s);
    if (err == hipSuccess)
      err = hipMemcpyAsync(sums, d_out, sizeof(sums), hipMemcpyDeviceToHost, s);
    if (err == hipSuccess) err = hipStreamSynchronize(s);
    return err;
  };
  double phi[4] = {phi_init[0], phi_init[1], phi_init[2], phi_init[3]};
  double c[3] = {0.0, 0.0, 0.0}, cost_sse = 0.0;
  int iters = 0, converged = 0;
  if (e == hipSuccess) e = eval(phi, 1, nullptr);
  bool cost_ok = false;
  if (e == hipSuccess) {
    // cost: normal equations of the affine model
    double M[9], r[3] = {sums[21], sums[22], sums[23]};
    unpack_sym(3, sums + 15, M);
    cost_ok = solve_small(3, M, r, c);
    // the residuals summed directly (the normal-equation form cancels badly)
    e = eval(phi, 2, c);
    cost_sse = cost_ok ? sums[24] : 0.0;
  }
  if (e == hipSuccess) {
    // gain: Levenberg-Marquardt with Marquardt's diagonal scaling
    double F = sums[0], H[16], g[4];
    unpack_sym(4, sums + 1, H);
    for (int k = 0; k < 4; ++k) g[k] = sums[11 + k];
    double lam = 1e-3;
    while (iters < max_iter && e == hipSuccess) {
      ++iters;
      double A[16], b[4], d[4];
      std::memcpy(A, H, sizeof A);
      for (int k = 0; k < 4; ++k) {
        A[k * 4 + k] += lam * (H[k * 4 + k] > 1e-300 ? H[k * 4 + k] : 1e-300);
        b[k] = -g[k];
      }
      if (!solve_small(4, A, b, d)) break;   // singular: every tau clamped, or no data
      double trial[4];
      for (int k = 0; k < 4; ++k) trial[k] = phi[k] + d[k];
      e = eval(trial, 0, nullptr);
      if (e != hipSuccess) break;
      if (sums[0] < F) {
        const double rel = (F - sums[0]) / (F > 0.0 ? F : 1.0);
        std::memcpy(phi, trial, sizeof phi);
        F = sums[0];
        unpack_sym(4, sums + 1, H);
        for (int k = 0; k < 4; ++k) g[k] = sums[11 + k];
        lam = lam / 10.0 > 1e-15 ? lam / 10.0 : 1e-15;
        double step = 0.0, size = 0.0;
        for (int k = 0; k < 4; ++k) {
          step += d[k] * d[k];
          size += phi[k] * phi[k];
        }
        if (rel < 1e-15 || step <= 1e-24 * (1.0 + size)) {
          converged = 1;
          break;
        }
      } else {
        lam *= 10.0;
        if (lam > 1e16) {
          converged = 1;   // no descent left at machine precision
          break;
        }
      }
    }
    if (stats) {
      stats[0] = F;
      stats[1] = cost_sse;
      stats[2] = iters;
      stats[3] = converged;
    }
  }
  (void)hipFree(d_budgets);
  (void)hipFree(d_part);
  (void)hipFree(d_out);
  if (e != hipSuccess) return hip_fail(e, "graft_saba_fit");
  for (int k = 0; k < 4; ++k) phi_out[k] = static_cast<float>(phi[k]);
  for (int k = 0; k < 3; ++k) c_out[k] = static_cast<float>(c[k]);
  return GRAFT_OK;
}

int64_t graft_tdes_param_count(const graft_tdes_dims *d) {
  if (!d || d->emb_dim < 1 || d->score_dim < 1 || d->num_pos < 1) return -1;
  return 2 * static_cast<int64_t>(d->emb_dim) * d->score_dim +
         static_cast<int64_t>(d->num_pos) * d->score_dim + 1;
}

int graft_tdes_create(const graft_tdes_dims *dims, graft_tdes **out) {
  if (!dims || !out) return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_create: NULL argument");
  *out = nullptr;
  const graft_tdes_dims d = *dims;
  if (d.vocab < 1 || d.emb_dim < 1 || d.score_dim < 1 || d.num_pos < 1 || d.top_k < 1 ||
      d.max_groups < 0 || d.max_pairs < 0)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_create: sizes must be positive");
  if (d.top_k > d.vocab)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_create: top_k %d > vocab %d", d.top_k, d.vocab);
  if (!graft::tdes_shape_supported(d.emb_dim, d.score_dim, d.num_pos, d.top_k))
    return fail(GRAFT_ERR_UNSUPPORTED,
                "graft_tdes_create: unsupported shape E=%d m=%d L=%d K=%d (E in {32, 64, 128}, "
                "E*M <= 4096, L*M <= 1024 for M = m rounded up to 16, K <= 64)",
                d.emb_dim, d.score_dim, d.num_pos, d.top_k);
  if (static_cast<int64_t>(d.max_groups) * d.top_k > (int64_t{1} << 31) - 1)
    return fail(GRAFT_ERR_UNSUPPORTED, "graft_tdes_create: max_groups * top_k too large");
  graft_tdes *t = new (std::nothrow) graft_tdes();
  if (!t) return fail(GRAFT_ERR_OUT_OF_MEMORY, "graft_tdes_create: host allocation failed");
  t->dims = d;
  const graft::TdesWorkspace ws = graft::tdes_workspace(d);
  hipError_t e = dalloc(&t->dyc, static_cast<size_t>(ws.dyc));
  if (e == hipSuccess) e = dalloc(&t->dyp, static_cast<size_t>(ws.dyp));
  if (e == hipSuccess) e = dalloc(&t->part_u, static_cast<size_t>(ws.part_u));
  if (e == hipSuccess) e = dalloc(&t->part_d, static_cast<size_t>(ws.part_d));
  if (e == hipSuccess) e = dalloc(&t->part_w, static_cast<size_t>(ws.part_w));
  if (e == hipSuccess) e = dalloc(&t->error_flag, 1);
  if (e == hipSuccess) e = hipMemset(t->error_flag, 0, sizeof(uint32_t));
  if (e != hipSuccess) {
    graft_tdes_destroy(t);
    return e == hipErrorOutOfMemory ? fail(GRAFT_ERR_OUT_OF_MEMORY, "graft_tdes_create: %s",
                                           hipGetErrorString(e))
                                    : hip_fail(e, "graft_tdes_create");
  }
  *out = t;
  return GRAFT_OK;
}

void graft_tdes_destroy(graft_tdes *t) {
  if (!t) return;
  (void)hipDeviceSynchronize();
  (void)hipFree(t->dyc);
  (void)hipFree(t->dyp);
  (void)hipFree(t->part_u);
  (void)hipFree(t->part_d);
  (void)hipFree(t->part_w);
  (void)hipFree(t->error_flag);
  delete t;
}

int graft_tdes_step(graft_tdes *t, const float *emb, const graft_tdes_batch *b,
                    const graft_tdes_hyper *h, int32_t step, float *theta, float *adam_m,
                    float *adam_v, double *loss, float *grad, graft_stream_t stream) {
  if (!t || !emb || !b || !h || !theta || !adam_m || !adam_v)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: NULL argument");
  const graft_tdes_dims &d = t->dims;
  if (b->n_groups < 0 || b->n_groups > d.max_groups)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: n_groups %d outside 0..%d", b->n_groups,
                d.max_groups);
  if (b->n_pairs < 0 || b->n_pairs > d.max_pairs)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: n_pairs %d outside 0..%d", b->n_pairs,
                d.max_pairs);
  if (b->n_groups > 0 &&
      (!b->parent || !b->depth || !b->child || !b->logq || !b->z_target || !b->target))
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: a group array is NULL");
  if (b->n_pairs > 0 && !b->pairs)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: pairs is NULL");
  if (reinterpret_cast<uintptr_t>(emb) % 16 != 0 || reinterpret_cast<uintptr_t>(theta) % 16 != 0)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: emb and theta must be 16-byte aligned");
  if (step < 1) return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: step must be >= 1");
  const float hv[10] = {h->lambda_kl, h->lambda_pair, h->lambda_bce, h->gamma, h->w1,
                        h->lr, h->weight_decay, h->beta1, h->beta2, h->eps};
  for (float v : hv)
    if (!std::isfinite(v)) return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: non-finite hyper-parameter");
  if (h->lr < 0.0f || h->weight_decay < 0.0f || h->eps <= 0.0f || h->beta1 < 0.0f ||
      h->beta1 >= 1.0f || h->beta2 < 0.0f || h->beta2 >= 1.0f)
    return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_step: AdamW settings out of range");
  hipError_t e = graft::launch_tdes_step(t, emb, b, h, step, theta, adam_m, adam_v, loss, grad,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "graft_tdes_step");
  return GRAFT_OK;
}

int graft_tdes_device_status(graft_tdes *t, graft_stream_t stream) {
  if (!t) return fail(GRAFT_ERR_INVALID_ARG, "graft_tdes_device_status: NULL trainer");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint32_t flag = 0;
  hipError_t e = hipMemcpyAsync(&flag, t->error_flag, sizeof flag, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "graft_tdes_device_status");
  if (flag) {
    e = hipMemsetAsync(t->error_flag, 0, sizeof flag, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "graft_tdes_device_status: clear");
    return fail(GRAFT_ERR_DEVICE_DATA, "training step dropped items with invalid ids (flags 0x%x)",
                flag);
  }
  return GRAFT_OK;
}

}  // extern "C"
