// k_scorer.hip -- TDES edge scoring (Sec. "Target-Distilled Edge Scoring").
//
// projection_kernel: the cached projections g_p(e) = e^T G_p and g_c(e) =
//   e^T G_c of every vocabulary token, computed once per scorer; the paper notes
//   they depend only on the token id.  fp64 accumulation, fp32 storage.
// edge_kernel: for one (sequence, depth) it gathers the projections of the K
//   children and of the parents (the root token at depth 1, else the K
//   candidates of the previous depth) into LDS, forms every parent-child dot
//   product (eq. tdes-bitower), centers over the children of each parent when
//   asked (eq. tdes-center) and adds log q of the child (eq. tdes-score).
//   Selection's copy of the scores is indexed by token-id rank: row (depth,
//   rank of the parent's id) holds the K children in the order of their ids,
//   so selection appends a parent's children in canonical order by filtering
//   the row against its threshold, with no ranking; the exported table keeps
//   the candidates' logit-rank order.
// The K x m x K contraction of a (sequence, depth), at most 64 x 64 x 64, runs
// on fp32 matrix cores in 16 x 16 tiles (edge_tiles); the depth-1 block of
// each sequence also computes its SABA budget.
#include "graft_internal.h"
#include "edge_mfma.h"
#include "saba_device.h"

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
constexpr int kGather = 8;         // projection loads (16 bytes) in flight per lane

// Division by a runtime divisor d <= 64 of numerators n below 2^26, without a
// branch: the high half of n * ceil(2^32 / d) in 64 bits.  Exact in that
// range: with ceil(2^32 / d) = (2^32 + e) / d, 0 <= e < d, the quotient is
// n / d plus n e / (d 2^32) < 2^-6 <= 1/d, which never reaches the next
// integer.
struct FastDiv {
  uint64_t m;
  __device__ __forceinline__ uint32_t div(uint32_t n) const {
    return static_cast<uint32_t>((static_cast<uint64_t>(n) * m) >> 32);
  }
};
FastDiv make_fastdiv(uint32_t d) { return FastDiv{((1ull << 32) + d - 1) / d}; }

// One wave per (sequence b, depth l).  Dynamic LDS: parents [K][mp],
// children [K][mp] (rows of m floats padded to a multiple of 4 plus 4: 16-byte
// aligned rows that start on different banks), depth embedding [m], log q [K],
// token ids [K], their ranks by id [K], clamped child and parent ids [K],
// parent tokens [K] and their ranks by id [K].  The scores come from
// edge_tiles<MK, NT> when m = 4 MK is a multiple of 16 (NT column tiles of
// 16 children), else from edge_passes<KQ> (KQ >= ceil(m / 4)).
template <int MK, int NT, int KQ>
__global__ void __launch_bounds__(kEdgeThreads)
edge_kernel(int L, int K, int m, int64_t V, FastDiv mdiv4, const int32_t *__restrict__ topk_ids,
            const float *__restrict__ topk_logq, const int32_t *__restrict__ root_token,
            const float *__restrict__ P, const float *__restrict__ Q,
            const float *__restrict__ depth_emb, ScorerParams sp,
            float *__restrict__ edge_rows, int32_t *__restrict__ cand_by_rank,
            uint8_t *__restrict__ positive,
            float *__restrict__ edge_out, uint32_t *__restrict__ error_flag, SabaArgs sa,
            SabaParams sp_saba) {
  extern __shared__ float smem[];
  const int mp = ((m + 3) & ~3) + 4;
  float *s_par = smem;
  float *s_chd = s_par + K * mp;
  float *s_u = s_chd + K * mp;           // 16-byte aligned
  float *s_lq = s_u + m;
  int32_t *s_tok = reinterpret_cast<int32_t *>(s_lq + K);
  int32_t *s_idr = s_tok + K;
  int32_t *s_cid = s_idr + K;
  int32_t *s_pid = s_cid + K;
  int32_t *s_ptok = s_pid + K;     // parent tokens (depth >= 2)
  int32_t *s_pidr = s_ptok + K;    // rank of each parent's token id in its depth

  // depth-major blocks: with a batch that is a multiple of the 8 XCDs, every
  // depth of sequence b runs on the XCD that the select block of b (block b)
  // runs on, so selection's reads of the rows find them in that XCD's L2
  const int batch = static_cast<int>(gridDim.x) / L;
  const int b = blockIdx.x % batch;
  const int l = blockIdx.x / batch;
  const int n_par = (l == 0) ? 1 : K;
  const int64_t row = static_cast<int64_t>(b) * L + l;
  const int lane = threadIdx.x;
  SabaIn saba_in{};
  if (l == 0) saba_in = saba_load(sa, sp_saba, b, L);

  int32_t root = root_token[b];
  if (root < 0 || root >= V) {
    if (lane == 0) atomicOr(error_flag, 1u);
    root = 0;
  }
  // token ids (clamped copies for the gathers; ids fall outside [0, V) only
  // with non-finite logits), log q and the depth embedding
  if (lane < K) {
    const int32_t ct = topk_ids[row * K + lane];
    const int32_t pt = (l == 0) ? root : topk_ids[(row - 1) * K + lane];
    s_tok[lane] = ct;
    s_lq[lane] = topk_logq[row * K + lane];
    s_cid[lane] = (ct < 0 || ct >= V) ? 0 : ct;
    s_pid[lane] = (pt < 0 || pt >= V) ? 0 : pt;
    s_ptok[lane] = pt;
  }
  for (int j = lane; j < m; j += kEdgeThreads) s_u[j] = sp.has_depth_emb ? depth_emb[l * m + j] : 0.f;
  __syncthreads();
  // rank of each candidate's token id within the depth
  if (lane < K) {
    const int32_t tc = s_tok[lane];
    int r = 0;
#pragma unroll 8
    for (int c2 = 0; c2 < K; ++c2) r += s_tok[c2] < tc;
    s_idr[lane] = r;
    cand_by_rank[row * K + r] = tc;
    int rp = 0;
    if (l > 0) {
      const int32_t tp = s_ptok[lane];
#pragma unroll 8
      for (int c2 = 0; c2 < K; ++c2) rp += s_ptok[c2] < tp;
    }
    s_pidr[lane] = rp;
  }
  // projections of children and parents plus the depth embedding, 16 bytes a
  // load when m % 4 == 0; every load of a batch is issued before any store
  if ((m & 3) == 0) {
    const int m4 = m >> 2;
    const int nq = K * m4, total = nq + n_par * m4;
    for (int base = 0; base < total; base += kGather * kEdgeThreads) {
      // the batch's token ids first (LDS), then its projection loads
      int32_t tok[kGather], j4s[kGather];
      bool child[kGather];
#pragma unroll
      for (int k = 0; k < kGather; ++k) {
        int t = base + k * kEdgeThreads + lane;
        t = t < total ? t : total - 1;
        child[k] = t < nq;
        const int tt = child[k] ? t : t - nq;
        const int r = static_cast<int>(mdiv4.div(static_cast<uint32_t>(tt)));
        j4s[k] = tt - r * m4;
        tok[k] = child[k] ? s_cid[r] : s_pid[r];
      }
      float4 v[kGather];
#pragma unroll
      for (int k = 0; k < kGather; ++k) {
        const float *src = (child[k] ? Q : P) + static_cast<int64_t>(tok[k]) * m;
        v[k] = reinterpret_cast<const float4 *>(src)[j4s[k]];
      }
#pragma unroll
      for (int k = 0; k < kGather; ++k) {
        const int t = base + k * kEdgeThreads + lane;
        if (t >= total) continue;
        const int tt = t < nq ? t : t - nq;
        const int r = static_cast<int>(mdiv4.div(static_cast<uint32_t>(tt))), j4 = tt - r * m4;
        const float4 u = reinterpret_cast<const float4 *>(s_u)[j4];
        float4 *dst = reinterpret_cast<float4 *>((t < nq ? s_chd : s_par) + r * mp) + j4;
        *dst = make_float4(v[k].x + u.x, v[k].y + u.y, v[k].z + u.z, v[k].w + u.w);
      }
    }
  } else {
    const int nq = K * m, total = nq + n_par * m;
    for (int t = lane; t < total; t += kEdgeThreads) {
      const int tt = t < nq ? t : t - nq;
      const int r = tt / m, j = tt % m;
      const float *src = t < nq ? Q + static_cast<int64_t>(s_cid[r]) * m
                                : P + static_cast<int64_t>(s_pid[r]) * m;
      (t < nq ? s_chd : s_par)[r * mp + j] = src[j] + s_u[j];
    }
  }
  __syncthreads();

  const float fscale = sp.scale / sqrtf(static_cast<float>(m));
  const int64_t base = row * K * K;
  // selection's copy is indexed by token-id rank (parent row, child column);
  // the exported table keeps the candidates' rank order
  const int32_t *prank = l == 0 ? nullptr : s_pidr;
  float *out = edge_out ? edge_out + base : nullptr;
  bool pos;
  if constexpr (MK > 0) {
    if (n_par > 16) {
      // the parents in two halves of whole 16-row tiles, their chains interleaved
      const int h = ((n_par + 31) / 32) * 16;
      const EdgeJob job[2] = {
          {s_par, s_chd, h, s_lq, s_idr, prank, edge_rows + base, out},
          {s_par + h * mp, s_chd, n_par - h, s_lq, s_idr, prank + h, edge_rows + base,
           out ? out + h * K : nullptr}};
      pos = edge_tiles<MK, NT, 2>(job, mp, K, fscale, sp.beta, sp.center);
    } else {
      const EdgeJob job[1] = {{s_par, s_chd, n_par, s_lq, s_idr, prank, edge_rows + base, out}};
      pos = edge_tiles<MK, NT, 1>(job, mp, K, fscale, sp.beta, sp.center);
    }
  } else
    pos = edge_passes<KQ>(s_par, s_chd, mp, n_par, K, m, fscale, sp.beta, sp.center, s_lq, s_idr,
                          prank, edge_rows + base, out);
  if (edge_out && l == 0)
    for (int i = K + lane; i < K * K; i += kEdgeThreads) edge_out[base + i] = 0.f;
  const bool any_pos = __ballot(pos) != 0ull;
  if (lane == 0) positive[row] = any_pos ? 1 : 0;
  // the depth-1 block (one parent, the lightest) also computes the budget
  if (l == 0) saba_budget(sa, sp_saba, b, L, saba_in);
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

hipError_t launch_edge_scores(graft_ctx *ctx, const RoundScratch &ws, const graft_round_in *in,
                              const graft_tree_out *out, hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  const int batch = in->batch;
  const int32_t *root_token = in->root_token;
  float *edge_out = out->edge_scores;
  const SabaArgs sa = saba_args(ctx, ws, in, out);
  const int K = d.top_k, m = ctx->scorer.score_dim;
  const size_t mp = ((m + 3) & ~3) + 4;
  const size_t lds = sizeof(float) * (2 * static_cast<size_t>(K) * mp + K + m) +
                     sizeof(int32_t) * 6 * K;
  const FastDiv mdiv4 = make_fastdiv(static_cast<uint32_t>(m >= 4 ? m / 4 : 1));
  const dim3 grid(batch * d.num_pos), block(kEdgeThreads);
#define GRAFT_EDGE(MK, NT, KQ)                                                                 \
  hipLaunchKernelGGL((edge_kernel<MK, NT, KQ>), grid, block, lds, stream, d.num_pos, K, m,   \
                     static_cast<int64_t>(d.vocab), mdiv4, ws.topk_ids, ws.topk_logq,       \
                     root_token, ctx->proj_parent, ctx->proj_child, ctx->depth_emb,           \
                     ctx->scorer, ws.edge_rows, ws.cand_by_rank,                            \
                     ws.positive, edge_out, ctx->error_flag, sa, ctx->saba)
#define GRAFT_EDGE_TILES(MK)                                                                   \
  do {                                                                                         \
    if (K <= 16) GRAFT_EDGE(MK, 1, 0);                                                         \
    else if (K <= 32) GRAFT_EDGE(MK, 2, 0);                                                    \
    else GRAFT_EDGE(MK, 4, 0);                                                                 \
  } while (0)
  // matrix-core tiles when m is a multiple of 16, else VALU passes with
  // ceil(m / 4) groups of four per row
  const int mk = (m + 3) / 4;
  if (m == 16) GRAFT_EDGE_TILES(4);
  else if (m == 32) GRAFT_EDGE_TILES(8);
  else if (m == 48) GRAFT_EDGE_TILES(12);
  else if (m == 64) GRAFT_EDGE_TILES(16);
  else if (mk <= 2) GRAFT_EDGE(0, 1, 2);
  else if (mk <= 4) GRAFT_EDGE(0, 1, 4);
  else if (mk <= 8) GRAFT_EDGE(0, 1, 8);
  else GRAFT_EDGE(0, 1, 16);
#undef GRAFT_EDGE_TILES
#undef GRAFT_EDGE
  return hipGetLastError();
}

}  // namespace graft
