// k_select.hip -- SABA budget, budgeted best-first selection, canonical
// emission and the ancestor mask; one workgroup per sequence.
//
// SABA (Sec. "State-Aware Budget Allocation"): tau = max(phi . [1, conf, ent,
//   hist], tau_min); U(B) = (1 - exp(-B/tau)) / (c0 + c1 B + c2 B prefix)
//   (eqs. saba-gain, saba-cost) is evaluated for every grid budget by one lane
//   each in fp64; B_t = the smallest budget with the largest U
//   (eq. saba-objective).
// Selection (DDTree paragraph; TDES "Inference", eq. tdes-path-score): the
//   candidate prefixes are ranked by their path score, the fp64 sum of fp32
//   edge scores from the root, in a max-heap; the best prefix is popped until
//   N = min(B_t, N_max) nodes are selected or no prefix is left.  Expansion is
//   lazy: popping the r-th best child of a parent pushes that parent's
//   (r+1)-th child and the popped node's best child.  Because each parent's
//   children were ranked by edge score (ties: token id), this pops exactly the
//   prefixes an eager push-all-children heap pops, with a frontier of at most
//   N + 1 entries.
// Emission: canonical numbering (depth ascending, token path ascending),
//   token ids, parent indices, position ids base_pos + depth, path scores, and
//   the ancestor-or-self bitset rows.
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kSelThreads = 256;

struct SelectArgs {
  int L, K, n_max, words, window;
  const float *row_stats;       // [B, L, 3]
  const float *sorted_score;    // [B, L, K, K]
  const uint8_t *sorted_child;  // [B, L, K, K]
  const int32_t *topk_ids;      // [B, L, K]
  const int32_t *root_token, *base_pos, *prefix_len, *fixed_budget;
  const float *hist;
  const int32_t *hist_ring;     // [B, window] (used when hist == nullptr)
  int32_t *budget, *n_nodes, *tokens, *parents, *pos_ids;
  uint64_t *mask;
  double *node_scores;
  float *saba_state;
};

// frontier entry info: parent node + 1 (11 bits) | rank (6) | slot (6) | depth-1 (6)
__device__ __forceinline__ int32_t pack_info(int parent, int rank, int slot, int depth) {
  return ((parent + 1) << 18) | (rank << 12) | (slot << 6) | (depth - 1);
}
__device__ __forceinline__ int info_parent(int32_t v) { return (v >> 18) - 1; }
__device__ __forceinline__ int info_rank(int32_t v) { return (v >> 12) & 63; }
__device__ __forceinline__ int info_slot(int32_t v) { return (v >> 6) & 63; }
__device__ __forceinline__ int info_depth(int32_t v) { return (v & 63) + 1; }

struct SelShared {
  double h_score[kMaxNodes + 1];
  int32_t h_info[kMaxNodes + 1];
  int32_t h_tok[kMaxNodes + 1];
  double n_score[kMaxNodes];
  int32_t n_parent[kMaxNodes];
  int32_t n_depth[kMaxNodes];
  int32_t n_slot[kMaxNodes];
  int32_t n_tok[kMaxNodes];
  int32_t canon[kMaxNodes];   // pop index -> canonical index
  int32_t cpar[kMaxNodes];    // canonical parents
  double saba_u[kMaxGrid];
  int32_t n_sel;
  int32_t budget;
  int32_t max_depth;
};

// Is frontier entry a ranked before entry b?  (score desc, depth asc, path asc)
__device__ bool ranks_before(const SelShared &s, int a, int b) {
  const double sa = s.h_score[a], sb = s.h_score[b];
  if (sa != sb) return sa > sb;
  const int da = info_depth(s.h_info[a]), db = info_depth(s.h_info[b]);
  if (da != db) return da < db;
  // same depth: compare token paths; walk both parent chains up to their
  // common ancestor, the tokens just below it decide
  int ta = s.h_tok[a], tb = s.h_tok[b];
  int x = info_parent(s.h_info[a]), y = info_parent(s.h_info[b]);
  while (x != y) {
    ta = s.n_tok[x];
    tb = s.n_tok[y];
    x = s.n_parent[x];
    y = s.n_parent[y];
  }
  return ta < tb;
}

__device__ void heap_swap(SelShared &s, int i, int j) {
  const double sc = s.h_score[i];
  s.h_score[i] = s.h_score[j];
  s.h_score[j] = sc;
  const int32_t in = s.h_info[i];
  s.h_info[i] = s.h_info[j];
  s.h_info[j] = in;
  const int32_t tk = s.h_tok[i];
  s.h_tok[i] = s.h_tok[j];
  s.h_tok[j] = tk;
}

__device__ void heap_push(SelShared &s, int &n, double score, int32_t info, int32_t tok) {
  int i = n++;
  s.h_score[i] = score;
  s.h_info[i] = info;
  s.h_tok[i] = tok;
  while (i > 0) {
    const int p = (i - 1) >> 1;
    if (!ranks_before(s, i, p)) break;
    heap_swap(s, i, p);
    i = p;
  }
}

__device__ void heap_pop_root(SelShared &s, int &n) {
  --n;
  if (n == 0) return;
  s.h_score[0] = s.h_score[n];
  s.h_info[0] = s.h_info[n];
  s.h_tok[0] = s.h_tok[n];
  int i = 0;
  for (;;) {
    const int l = 2 * i + 1, r = l + 1;
    int best = i;
    if (l < n && ranks_before(s, l, best)) best = l;
    if (r < n && ranks_before(s, r, best)) best = r;
    if (best == i) break;
    heap_swap(s, i, best);
    i = best;
  }
}

__global__ void __launch_bounds__(kSelThreads) select_kernel(SelectArgs a, SabaParams sp, int use_saba) {
  __shared__ SelShared s;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int L = a.L, K = a.K;

  // ---------------- SABA (wave 0) ----------------
  if (tid < kWave) {
    double hist;
    if (a.hist) {
      hist = static_cast<double>(a.hist[b]);
    } else {
      int64_t sum = 0;
      for (int i = 0; i < a.window; ++i) sum += a.hist_ring[b * a.window + i];
      hist = static_cast<double>(sum) / static_cast<double>(a.window);
    }
    double conf = 0.0, ent = 0.0;
    for (int l = 0; l < L; ++l) {
      conf += static_cast<double>(a.row_stats[(static_cast<int64_t>(b) * L + l) * 3 + 1]);
      ent += static_cast<double>(a.row_stats[(static_cast<int64_t>(b) * L + l) * 3 + 2]);
    }
    conf /= static_cast<double>(L);
    ent /= static_cast<double>(L);
    double tau = 0.0;
    int budget;
    if (use_saba) {
      tau = static_cast<double>(sp.phi[0]) + static_cast<double>(sp.phi[1]) * conf +
            static_cast<double>(sp.phi[2]) * ent + static_cast<double>(sp.phi[3]) * hist;
      if (tau < static_cast<double>(sp.tau_min)) tau = static_cast<double>(sp.tau_min);
      const double prefix = a.prefix_len ? static_cast<double>(a.prefix_len[b]) : 0.0;
      if (tid < sp.n_grid) {
        const double B = static_cast<double>(sp.grid[tid]);
        s.saba_u[tid] = (1.0 - exp(-B / tau)) /
                        (static_cast<double>(sp.c0) + static_cast<double>(sp.c1) * B +
                         static_cast<double>(sp.c2) * B * prefix);
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
      budget = sp.grid[0];
      double ub = s.saba_u[0];
      for (int i = 1; i < sp.n_grid; ++i)
        if (s.saba_u[i] > ub) {
          ub = s.saba_u[i];
          budget = sp.grid[i];
        }
    } else {
      budget = a.fixed_budget[b];
    }
    if (tid == 0) {
      s.budget = budget;
      a.budget[b] = budget;
      if (a.saba_state) {
        a.saba_state[b * 4 + 0] = static_cast<float>(conf);
        a.saba_state[b * 4 + 1] = static_cast<float>(ent);
        a.saba_state[b * 4 + 2] = static_cast<float>(hist);
        a.saba_state[b * 4 + 3] = static_cast<float>(tau);
      }
    }
  }
  __syncthreads();

  // ---------------- best-first selection (one thread) ----------------
  const float *ss = a.sorted_score + static_cast<int64_t>(b) * L * K * K;
  const uint8_t *sc = a.sorted_child + static_cast<int64_t>(b) * L * K * K;
  const int32_t *cand = a.topk_ids + static_cast<int64_t>(b) * L * K;
  if (tid == 0) {
    int n_target = s.budget < a.n_max ? s.budget : a.n_max;
    if (n_target < 0) n_target = 0;
    int hn = 0, n_sel = 0, max_depth = 0;
    if (n_target > 0) {
      const int c0 = sc[0];
      heap_push(s, hn, static_cast<double>(ss[0]), pack_info(-1, 0, c0, 1), cand[c0]);
    }
    while (n_sel < n_target && hn > 0) {
      const double score = s.h_score[0];
      const int32_t info = s.h_info[0];
      const int32_t tok = s.h_tok[0];
      heap_pop_root(s, hn);
      const int p = info_parent(info), r = info_rank(info), slot = info_slot(info);
      const int d = info_depth(info);
      const int i = n_sel++;
      s.n_score[i] = score;
      s.n_parent[i] = p;
      s.n_depth[i] = d;
      s.n_slot[i] = slot;
      s.n_tok[i] = tok;
      if (d > max_depth) max_depth = d;
      // next sibling under the same parent
      if (r + 1 < K) {
        const int pslot = p < 0 ? 0 : s.n_slot[p];
        const double pscore = p < 0 ? 0.0 : s.n_score[p];
        const int64_t off = (static_cast<int64_t>(d - 1) * K + pslot) * K + (r + 1);
        const int cs = sc[off];
        heap_push(s, hn, pscore + static_cast<double>(ss[off]), pack_info(p, r + 1, cs, d),
                  cand[(d - 1) * K + cs]);
      }
      // best child of the new node
      if (d < L) {
        const int64_t off = (static_cast<int64_t>(d) * K + slot) * K;
        const int cs = sc[off];
        heap_push(s, hn, score + static_cast<double>(ss[off]), pack_info(i, 0, cs, d + 1),
                  cand[d * K + cs]);
      }
    }
    s.n_sel = n_sel;
    s.max_depth = max_depth;
    a.n_nodes[b] = n_sel;
  }
  __syncthreads();

  // ---------------- canonical numbering ----------------
  const int n = s.n_sel;
  int offset = 0;
  for (int dd = 1; dd <= s.max_depth; ++dd) {
    for (int i = tid; i < n; i += kSelThreads) {
      if (s.n_depth[i] != dd) continue;
      const int pi = s.n_parent[i];
      const uint64_t key = (static_cast<uint64_t>(pi < 0 ? 0 : s.canon[pi] + 1) << 32) |
                           static_cast<uint32_t>(s.n_tok[i]);
      int rank = 0;
      for (int j = 0; j < n; ++j) {
        if (s.n_depth[j] != dd) continue;
        const int pj = s.n_parent[j];
        const uint64_t kj = (static_cast<uint64_t>(pj < 0 ? 0 : s.canon[pj] + 1) << 32) |
                            static_cast<uint32_t>(s.n_tok[j]);
        rank += kj < key;
      }
      s.canon[i] = offset + rank;
    }
    __syncthreads();
    int cnt = 0;
    for (int j = 0; j < n; ++j) cnt += s.n_depth[j] == dd;
    offset += cnt;
  }

  // ---------------- emission ----------------
  const int64_t ob = static_cast<int64_t>(b) * a.n_max;
  const int32_t base = a.base_pos[b];
  for (int i = tid; i < a.n_max; i += kSelThreads) {
    if (i < n) {
      const int c = s.canon[i];
      const int pi = s.n_parent[i];
      const int cp = pi < 0 ? -1 : s.canon[pi];
      a.tokens[ob + c] = s.n_tok[i];
      a.parents[ob + c] = cp;
      a.pos_ids[ob + c] = base + s.n_depth[i];
      if (a.node_scores) a.node_scores[ob + c] = s.n_score[i];
      s.cpar[c] = cp;
    } else {
      a.tokens[ob + i] = -1;
      a.parents[ob + i] = -1;
      a.pos_ids[ob + i] = -1;
      if (a.node_scores) a.node_scores[ob + i] = 0.0;
    }
  }
  __syncthreads();

  // ---------------- ancestor mask ----------------
  if (a.mask) {
    uint64_t *mrow = a.mask + static_cast<int64_t>(b) * a.n_max * a.words;
    const int total = a.n_max * a.words;
    for (int idx = tid; idx < total; idx += kSelThreads) {
      const int r = idx / a.words, wd = idx % a.words;
      uint64_t bits = 0;
      if (r < n) {
        for (int j = r; j >= 0; j = s.cpar[j])
          if ((j >> 6) == wd) bits |= 1ull << (j & 63);
      }
      mrow[idx] = bits;
    }
  }
}

}  // namespace

hipError_t launch_select(graft_ctx *ctx, const graft_round_in *in, const graft_tree_out *out,
                         hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  SelectArgs a;
  a.L = d.num_pos;
  a.K = d.top_k;
  a.n_max = d.max_nodes;
  a.words = (d.max_nodes + 63) / 64;
  a.window = d.hist_window;
  a.row_stats = ctx->row_stats;
  a.sorted_score = ctx->sorted_score;
  a.sorted_child = ctx->sorted_child;
  a.topk_ids = ctx->topk_ids;
  a.root_token = in->root_token;
  a.base_pos = in->base_pos;
  a.prefix_len = in->prefix_len;
  a.fixed_budget = in->fixed_budget;
  a.hist = in->hist;
  a.hist_ring = ctx->hist_ring;
  a.budget = out->budget;
  a.n_nodes = out->n_nodes;
  a.tokens = out->tokens;
  a.parents = out->parents;
  a.pos_ids = out->pos_ids;
  a.mask = out->mask;
  a.node_scores = out->node_scores;
  a.saba_state = out->saba_state;
  const int use_saba = in->fixed_budget == nullptr;
  hipLaunchKernelGGL(select_kernel, dim3(in->batch), dim3(kSelThreads), 0, stream, a, ctx->saba,
                     use_saba);
  return hipGetLastError();
}

}  // namespace graft
