// k_scorer.hip -- TDES edge scoring (Sec. "Target-Distilled Edge Scoring").
//
// projection_kernel: the cached projections g_p(e) = e^T G_p and g_c(e) =
//   e^T G_c of every vocabulary token, computed once per scorer; the paper notes
//   they depend only on the token id.  fp64 accumulation, fp32 storage.
// edge_kernel: for one (sequence, depth) it gathers the projections of the K
//   children and of the parents (the root token at depth 1, else the K
//   candidates of the previous depth) into LDS, forms every parent-child dot
//   product (eq. tdes-bitower), centers over the children of each parent when
//   asked (eq. tdes-center) and adds log q of the child (eq. tdes-score).  It
//   then ranks the children of every parent by (score desc, token id asc) so
//   that selection can expand a parent's children lazily in order.
// The K x m x K contraction is at most 64 x 64 x 64 per (sequence, depth):
// VALU work on LDS-staged rows; there is no dense tile to feed MFMA.
#include "graft_internal.h"

namespace graft {
namespace {

__global__ void __launch_bounds__(256)
projection_kernel(const float *__restrict__ emb, const float *__restrict__ gp,
                  const float *__restrict__ gc, int64_t V, int E, int m,
                  float *__restrict__ P, float *__restrict__ Q) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= V * m) return;
  const int64_t v = idx / m;
  const int j = static_cast<int>(idx % m);
  const float *e = emb + v * E;
  double ap = 0.0, ac = 0.0;
  for (int i = 0; i < E; ++i) {
    const double x = static_cast<double>(e[i]);
    ap += x * static_cast<double>(gp[static_cast<int64_t>(i) * m + j]);
    ac += x * static_cast<double>(gc[static_cast<int64_t>(i) * m + j]);
  }
  P[idx] = static_cast<float>(ap);
  Q[idx] = static_cast<float>(ac);
}

constexpr int kEdgeThreads = 64;   // one wave per (sequence, depth)

// Dynamic LDS layout: parents [K][m+1], children [K][m+1] (rows padded by one
// float so that lanes reading different rows hit different banks), scores
// [K][K], row means [K], tokens [K].
__global__ void __launch_bounds__(kEdgeThreads)
edge_kernel(int L, int K, int m, int64_t V, const int32_t *__restrict__ topk_ids,
            const float *__restrict__ topk_logq, const int32_t *__restrict__ root_token,
            const float *__restrict__ P, const float *__restrict__ Q,
            const float *__restrict__ depth_emb, ScorerParams sp,
            float *__restrict__ sorted_score, uint8_t *__restrict__ sorted_child,
            uint8_t *__restrict__ id_rank, uint8_t *__restrict__ positive,
            float *__restrict__ edge_out, uint32_t *__restrict__ error_flag) {
  extern __shared__ float smem[];
  const int mp = m + 1;
  float *s_par = smem;
  float *s_chd = s_par + K * mp;
  float *s_score = s_chd + K * mp;
  float *s_mean = s_score + K * K;
  int32_t *s_tok = reinterpret_cast<int32_t *>(s_mean + K);

  const int b = blockIdx.x / L;
  const int l = blockIdx.x % L;
  const int n_par = (l == 0) ? 1 : K;
  const int64_t row = static_cast<int64_t>(b) * L + l;
  const int lane = threadIdx.x;

  int32_t root = root_token[b];
  if (root < 0 || root >= V) {
    if (lane == 0) atomicOr(error_flag, 1u);
    root = 0;
  }
  // stage projections (+ depth embedding) of parents and children
  for (int i = lane; i < K * m; i += kEdgeThreads) {
    const int c = i / m, j = i % m;
    const float u = sp.has_depth_emb ? depth_emb[l * m + j] : 0.f;
    int32_t ct = topk_ids[row * K + c];
    if (ct < 0 || ct >= V) ct = 0;   // only with non-finite logits
    s_chd[c * mp + j] = Q[static_cast<int64_t>(ct) * m + j] + u;
    if (c < n_par) {
      int32_t pt = (l == 0) ? root : topk_ids[(row - 1) * K + c];
      if (pt < 0 || pt >= V) pt = 0;
      s_par[c * mp + j] = P[static_cast<int64_t>(pt) * m + j] + u;
    }
  }
  for (int c = lane; c < K; c += kEdgeThreads) s_tok[c] = topk_ids[row * K + c];
  __syncthreads();

  // f(p, c) = s * <P[p] + u, Q[c] + u> / sqrt(m)
  const float fscale = sp.scale / sqrtf(static_cast<float>(m));
  for (int i = lane; i < n_par * K; i += kEdgeThreads) {
    const int p = i / K, c = i % K;
    const float *pv = s_par + p * mp, *cv = s_chd + c * mp;
    float acc = 0.f;
    for (int j = 0; j < m; ++j) acc = __builtin_fmaf(pv[j], cv[j], acc);
    s_score[i] = fscale * acc;
  }
  __syncthreads();
  for (int p = lane; p < n_par; p += kEdgeThreads) {
    float mean = 0.f;
    if (sp.center) {
      for (int c = 0; c < K; ++c) mean += s_score[p * K + c];
      mean /= static_cast<float>(K);
    }
    s_mean[p] = mean;
  }
  __syncthreads();
  // S = log q(c) + beta * (f - mean over the children of p)
  for (int i = lane; i < n_par * K; i += kEdgeThreads) {
    const int p = i / K, c = i % K;
    const float lq = topk_logq[row * K + c];
    s_score[i] = lq + sp.beta * (s_score[i] - s_mean[p]);
  }
  __syncthreads();
  // rank the children of each parent; write the ranked rows, the optional
  // table, the sign flag and the token-id rank of each candidate
  const int64_t base = row * K * K;
  bool pos = false;
  for (int i = lane; i < n_par * K; i += kEdgeThreads) {
    const int p = i / K, c = i % K;
    const float sc = s_score[i];
    const int32_t tc = s_tok[c];
    int rank = 0;
    for (int c2 = 0; c2 < K; ++c2) {
      const float o = s_score[p * K + c2];
      rank += (o > sc) || (o == sc && s_tok[c2] < tc);
    }
    sorted_score[base + p * K + rank] = sc;
    sorted_child[base + p * K + rank] = static_cast<uint8_t>(c);
    if (edge_out) edge_out[base + i] = sc;
    pos |= sc > 0.f;
  }
  if (edge_out && l == 0)
    for (int i = K + lane; i < K * K; i += kEdgeThreads) edge_out[base + i] = 0.f;
  for (int c = lane; c < K; c += kEdgeThreads) {
    int r = 0;
    for (int c2 = 0; c2 < K; ++c2) r += s_tok[c2] < s_tok[c];
    id_rank[row * K + c] = static_cast<uint8_t>(r);
  }
  const bool any_pos = __ballot(pos) != 0ull;
  if (lane == 0) positive[row] = any_pos ? 1 : 0;
}

}  // namespace

hipError_t launch_projection(graft_ctx *ctx, const graft_scorer_desc *d, hipStream_t stream) {
  const int64_t V = ctx->dims.vocab;
  const int m = d->score_dim;
  const int64_t n = V * m;
  const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
  hipLaunchKernelGGL(projection_kernel, dim3(blocks), dim3(256), 0, stream, d->emb, d->g_parent,
                     d->g_child, V, d->emb_dim, m, ctx->proj_parent, ctx->proj_child);
  return hipGetLastError();
}

hipError_t launch_edge_scores(graft_ctx *ctx, int batch, const int32_t *root_token,
                              float *edge_out, hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  const int K = d.top_k, m = ctx->scorer.score_dim;
  const size_t lds = sizeof(float) * (2 * static_cast<size_t>(K) * (m + 1) + K * K + K) +
                     sizeof(int32_t) * K;
  hipLaunchKernelGGL(edge_kernel, dim3(batch * d.num_pos), dim3(kEdgeThreads), lds, stream,
                     d.num_pos, K, m, static_cast<int64_t>(d.vocab), ctx->topk_ids,
                     ctx->topk_logq, root_token, ctx->proj_parent, ctx->proj_child,
                     ctx->depth_emb, ctx->scorer, ctx->sorted_score, ctx->sorted_child,
                     ctx->id_rank, ctx->positive, edge_out, ctx->error_flag);
  return hipGetLastError();
}

}  // namespace graft
