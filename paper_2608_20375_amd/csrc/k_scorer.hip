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
// The K x m x K contraction is at most 64 x 64 x 64 per (sequence, depth):
// VALU work, each lane keeping one child's projection in registers and
// reading the parents' rows from LDS as broadcasts; there is no dense tile to
// feed MFMA.  The depth-1 block of each sequence also computes its SABA
// budget.
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

// SABA inputs and outputs of one round (Sec. "State-Aware Budget Allocation").
struct SabaArgs {
  const float *row_stats;       // [B, L, 3]: lse, maxprob, entropy
  const float *hist;            // [B] caller's hist_t, or nullptr: the device ring
  const int32_t *hist_ring;     // [B, window]
  const int32_t *prefix_len;    // [B] or nullptr (0)
  const int32_t *fixed_budget;  // [B]: budgets given by the caller, or nullptr: SABA
  const float *adj_cos;         // [B, L - 1] adjacent hidden-state cosines, or nullptr
  int window;
  int32_t *budget;              // [B] out
  float *saba_state;            // [B, 4] out (conf, ent or degen, hist, tau) or nullptr
};

// B_t of sequence b by one wave: conf is the mean of the rows' top-1
// probability; the second feature is degen = mean_d r_d + (r_{L-1} - r_1)
// over the adjacent hidden-state cosines when they are given, else the mean
// row entropy standing in for it; hist is the caller's value or the ring's
// mean; tau = max(phi . [1, conf, feature, hist], tau_min); U(B) = (1 -
// exp(-B/tau)) / (c0 + c1 B + c2 B prefix) (eqs. saba-gain, saba-cost) for
// every grid budget, one lane each in fp64; B_t = the smallest budget with the
// largest U (eq. saba-objective).
// The budget's inputs, one wave's lanes; loaded before the edge work so that
// their latency overlaps it.
struct SabaIn {
  float f_conf, f_ent, f_r, f_hist;
  int32_t ring, prefix_i, fixed, grid;
};
__device__ __forceinline__ SabaIn saba_load(const SabaArgs &a, const SabaParams &sp, int b, int L) {
  const int lane = lane_id();
  SabaIn in;
  const float *rs = a.row_stats + (static_cast<int64_t>(b) * L + (lane < L ? lane : 0)) * 3;
  in.f_conf = rs[1];
  in.f_ent = rs[2];
  const int np = L - 1;
  in.f_r = (a.adj_cos && lane < np) ? a.adj_cos[static_cast<int64_t>(b) * np + lane] : 0.f;
  in.f_hist = a.hist ? a.hist[b] : 0.f;
  in.ring = (!a.hist && lane < a.window) ? a.hist_ring[static_cast<int64_t>(b) * a.window + lane] : 0;
  in.prefix_i = a.prefix_len ? a.prefix_len[b] : 0;
  in.fixed = a.fixed_budget ? a.fixed_budget[b] : 0;
  in.grid = lane < sp.n_grid ? sp.grid[lane] : 0;
  return in;
}

__device__ void saba_budget(const SabaArgs &a, const SabaParams &sp, int b, int L, const SabaIn &in) {
  const int lane = lane_id();
  const float f_conf = in.f_conf, f_ent = in.f_ent, f_r = in.f_r, f_hist = in.f_hist;
  const int32_t ring = in.ring, prefix_i = in.prefix_i, fixed = in.fixed, grid = in.grid;
  const int np = L - 1;
  double hist;
  if (a.hist) {
    hist = static_cast<double>(f_hist);
  } else {
    int64_t v = ring;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1)
      v += static_cast<int64_t>(xor_lane_u64(static_cast<uint64_t>(v), o));
    hist = static_cast<double>(v) / static_cast<double>(a.window);
  }
  double conf = lane < L ? static_cast<double>(f_conf) : 0.0;
  double ent = lane < L ? static_cast<double>(f_ent) : 0.0;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    conf += xor_lane_f64(conf, o);
    ent += xor_lane_f64(ent, o);
  }
  conf /= static_cast<double>(L);
  ent /= static_cast<double>(L);
  if (a.adj_cos) {
    // degen from the cosines r_1 .. r_{L-1} (lanes 0 .. L-2); 0 without a pair
    double r = lane < np ? static_cast<double>(f_r) : 0.0;
    const double r_first = static_cast<double>(__shfl(f_r, 0));
    const double r_last = static_cast<double>(__shfl(f_r, np > 0 ? np - 1 : 0));
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) r += xor_lane_f64(r, o);
    ent = np > 0 ? r / static_cast<double>(np) + (r_last - r_first) : 0.0;
  }
  double tau = 0.0;
  int budget;
  if (!a.fixed_budget) {
    tau = static_cast<double>(sp.phi[0]) + static_cast<double>(sp.phi[1]) * conf +
          static_cast<double>(sp.phi[2]) * ent + static_cast<double>(sp.phi[3]) * hist;
    if (tau < static_cast<double>(sp.tau_min)) tau = static_cast<double>(sp.tau_min);
    const double prefix = static_cast<double>(prefix_i);
    // the first maximum: largest U, ties (and a non-number U) to the smaller index
    double u = -INFINITY;
    if (lane < sp.n_grid) {
      const double B = static_cast<double>(grid);
      u = (1.0 - exp(-B / tau)) / (static_cast<double>(sp.c0) + static_cast<double>(sp.c1) * B +
                                   static_cast<double>(sp.c2) * B * prefix);
      if (!(u == u)) u = -INFINITY;
    }
    int best = lane;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const double ou = xor_lane_f64(u, o);
      const int ob = static_cast<int>(xor_lane(static_cast<uint32_t>(best), o));
      if (ou > u || (ou == u && ob < best)) {
        u = ou;
        best = ob;
      }
    }
    budget = __builtin_amdgcn_readlane(grid, best < sp.n_grid ? best : 0);
  } else {
    budget = fixed;
  }
  if (lane == 0) {
    a.budget[b] = budget;
    if (a.saba_state) {
      a.saba_state[b * 4 + 0] = static_cast<float>(conf);
      a.saba_state[b * 4 + 1] = static_cast<float>(ent);
      a.saba_state[b * 4 + 2] = static_cast<float>(hist);
      a.saba_state[b * 4 + 3] = static_cast<float>(tau);
    }
  }
}

// Sum over each run of SEG consecutive lanes, in every lane of the run.
template <int SEG>
__device__ __forceinline__ float seg_sum(float v) {
#pragma unroll
  for (int stride = 1; stride < SEG; stride <<= 1)
    v += __uint_as_float(xor_lane(__float_as_uint(v), stride));
  return v;
}

// One wave per (sequence b, depth l).  Dynamic LDS: parents [K][mp],
// children [K][mp] (rows of m floats padded to a multiple of 4 plus 4: 16-byte
// aligned rows that start on different banks), depth embedding [m], log q [K],
// token ids [K], their ranks by id [K], clamped child and parent ids [K],
// parent tokens [K] and their ranks by id [K].
// The (parent, child) pairs are processed SEG lanes per parent (SEG = K
// rounded up to a power of two), kRows = 64 / SEG parents at a time: lane c of
// a run keeps child c's row in registers, reads the parent's row from LDS (one
// address for the whole run), and forms the dot product, the centering over
// the parent's children and the score.  With m % 4 == 0 a row is KQ groups of
// four (KQ = m / 4 rounded up to a power of two; the child's groups past m / 4
// are zero), all of a parent row's loads issued before its products.
template <int SEG, int KQ>
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

  // per parent p (SEG lanes, child c = lane % SEG):
  //   f = s * <P[p] + u, Q[c] + u> / sqrt(m),  S = log q(c) + beta * (f - mean_c f)
  const float fscale = sp.scale / sqrtf(static_cast<float>(m));
  constexpr int kRows = kEdgeThreads / SEG;
  const int c = lane & (SEG - 1);
  const int cc = c < K ? c : 0;
  const int64_t base = row * K * K;
  bool pos = false;
  const int m4 = m >> 2;
  // the child's row, 16 bytes a register group (m % 4 == 0; groups past m / 4
  // hold zeros) or a float each
  float4 cr[KQ];
  if ((m & 3) == 0) {
    const float4 *c4 = reinterpret_cast<const float4 *>(s_chd + cc * mp);
#pragma unroll
    for (int q = 0; q < KQ; ++q) cr[q] = c4[q < m4 ? q : 0];
#pragma unroll
    for (int q = 0; q < KQ; ++q)
      if (q >= m4) cr[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const float lq = s_lq[cc];
  const int col = s_idr[cc];   // the child's column in selection's rows
  for (int p0 = 0; p0 < n_par; p0 += kRows) {
    const int p = p0 + lane / SEG;
    const bool valid = p < n_par && c < K;
    const int pp = p < n_par ? p : 0;
    const int prow = s_pidr[pp];
    const float *pv = s_par + pp * mp;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    if ((m & 3) == 0) {
      const float4 *p4 = reinterpret_cast<const float4 *>(pv);
      float4 x[KQ];
#pragma unroll
      for (int q = 0; q < KQ; ++q) x[q] = p4[q < m4 ? q : 0];
#pragma unroll
      for (int q = 0; q < KQ; ++q) {
        a0 = __builtin_fmaf(x[q].x, cr[q].x, a0);
        a1 = __builtin_fmaf(x[q].y, cr[q].y, a1);
        a2 = __builtin_fmaf(x[q].z, cr[q].z, a2);
        a3 = __builtin_fmaf(x[q].w, cr[q].w, a3);
      }
    } else {
      const float *cv = s_chd + cc * mp;
#pragma unroll 4
      for (int j = 0; j < m; ++j) a0 = __builtin_fmaf(pv[j], cv[j], a0);
    }
    const float f = fscale * ((a0 + a1) + (a2 + a3));
    float mean = 0.f;
    if (sp.center) mean = seg_sum<SEG>(valid ? f : 0.f) / static_cast<float>(K);
    const float S = (lq + sp.beta * (f - mean)) + 0.0f;   // -0 -> +0
    if (valid) {
      // selection's copy is indexed by token-id rank (parent row, child
      // column); the exported table keeps the candidates' rank order
      edge_rows[base + prow * K + col] = S;
      if (edge_out) edge_out[base + p * K + c] = S;
    }
    pos |= valid && S > 0.f;
  }
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
  SabaArgs sa;
  sa.row_stats = ws.row_stats;
  sa.hist = in->hist;
  sa.hist_ring = ctx->hist_ring;
  sa.prefix_len = in->prefix_len;
  sa.fixed_budget = in->fixed_budget;
  sa.adj_cos = in->hidden ? ws.adj_cos : nullptr;
  sa.window = d.hist_window;
  sa.budget = out->budget;
  sa.saba_state = out->saba_state;
  const int K = d.top_k, m = ctx->scorer.score_dim;
  const size_t mp = ((m + 3) & ~3) + 4;
  const size_t lds = sizeof(float) * (2 * static_cast<size_t>(K) * mp + K + m) +
                     sizeof(int32_t) * 6 * K;
  const FastDiv mdiv4 = make_fastdiv(static_cast<uint32_t>(m >= 4 ? m / 4 : 1));
  const dim3 grid(batch * d.num_pos), block(kEdgeThreads);
#define GRAFT_EDGE_KQ(SEG, KQ)                                                                 \
  hipLaunchKernelGGL((edge_kernel<SEG, KQ>), grid, block, lds, stream, d.num_pos, K, m,      \
                     static_cast<int64_t>(d.vocab), mdiv4, ws.topk_ids, ws.topk_logq,       \
                     root_token, ctx->proj_parent, ctx->proj_child, ctx->depth_emb,           \
                     ctx->scorer, ws.edge_rows, ws.cand_by_rank,                            \
                     ws.positive, edge_out, ctx->error_flag, sa, ctx->saba)
  // groups of four per score row (the scalar path, m % 4 != 0, takes 2)
  const int m4 = (m & 3) == 0 ? m / 4 : 0;
#define GRAFT_EDGE(SEG)                                                                        \
  do {                                                                                         \
    if (m4 <= 2) GRAFT_EDGE_KQ(SEG, 2);                                                        \
    else if (m4 <= 4) GRAFT_EDGE_KQ(SEG, 4);                                                   \
    else if (m4 <= 8) GRAFT_EDGE_KQ(SEG, 8);                                                   \
    else GRAFT_EDGE_KQ(SEG, 16);                                                               \
  } while (0)
  if (K <= 1) GRAFT_EDGE(1);
  else if (K <= 2) GRAFT_EDGE(2);
  else if (K <= 4) GRAFT_EDGE(4);
  else if (K <= 8) GRAFT_EDGE(8);
  else if (K <= 16) GRAFT_EDGE(16);
  else if (K <= 32) GRAFT_EDGE(32);
  else GRAFT_EDGE(64);
#undef GRAFT_EDGE
#undef GRAFT_EDGE_KQ
  return hipGetLastError();
}

}  // namespace graft
