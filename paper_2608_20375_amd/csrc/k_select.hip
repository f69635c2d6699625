// k_select.hip -- SABA budget, budgeted best-first selection, canonical
// emission and the ancestor mask; one workgroup per sequence.
//
// SABA (Sec. "State-Aware Budget Allocation"): tau = max(phi . [1, conf, ent,
//   hist], tau_min); U(B) = (1 - exp(-B/tau)) / (c0 + c1 B + c2 B prefix)
//   (eqs. saba-gain, saba-cost) is evaluated for every grid budget by one lane
//   each in fp64; B_t = the smallest budget with the largest U
//   (eq. saba-objective).
//
// Selection (DDTree paragraph; TDES "Inference", eq. tdes-path-score): prefixes
//   are ranked by their path score, the fp64 sum of fp32 edge scores from the
//   root, then by smaller depth, then by the smaller token path; best-first
//   pops the best prefix until N = min(B_t, N_max) nodes are selected.
//
//   When every edge score of the sequence is <= 0 a child never outranks its
//   parent, so the N prefixes best-first pops are exactly the N best prefixes
//   of the whole candidate trie.  The workgroup finds them in parallel:
//     pool  <- the K depth-1 prefixes
//     loop: keep the N best of the pool (exact selection: a 2048-bin
//           histogram of the scores locates the boundary bin, whose few
//           members are ranked with the full order); let theta be the N-th;
//           expand every kept prefix not yet expanded, adding only children
//           whose score reaches theta (a prefix of each parent's ranked row);
//           stop when every kept prefix is expanded.
//   A prefix outside the kept set can only gain better competitors, and a
//   skipped child is worse than theta, which only rises, so the result is the
//   exact top N.  Iterations <= depth of the tree + 1.
//   Otherwise (some positive edge score) one thread runs the heap directly.
//
// Emission: canonical numbering (depth ascending, token path ascending), token
//   ids, parent indices, position ids base_pos + depth, path scores, and the
//   ancestor-or-self bitset rows.
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kSelThreads = 512;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kPoolCap = 4096;
constexpr int kBins = 2048;

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

// Pool entry info: parent + 1 (13 bits) | depth - 1 (6) | slot (6) | expanded (1)
__device__ __forceinline__ int32_t pinfo(int parent, int depth, int slot, int expanded) {
  return (parent + 1) | ((depth - 1) << 13) | (slot << 19) | (expanded << 25);
}
__device__ __forceinline__ int pi_parent(int32_t v) { return (v & 0x1FFF) - 1; }
__device__ __forceinline__ int pi_depth(int32_t v) { return ((v >> 13) & 63) + 1; }
__device__ __forceinline__ int pi_slot(int32_t v) { return (v >> 19) & 63; }
__device__ __forceinline__ int pi_expanded(int32_t v) { return (v >> 25) & 1; }

struct SelMem {
  double p_score[kPoolCap];
  int32_t p_info[kPoolCap];
  int32_t map[kPoolCap];
  int32_t aux[kPoolCap + 1];
  int32_t hist[kBins + 1];
  int32_t pcnt[kBins + 1];
  int32_t cand[kMaxL * kMaxK];
  uint8_t idr[kMaxL * kMaxK];
  // serial heap (fallback)
  double h_score[kMaxNodes + 1];
  int32_t h_info[kMaxNodes + 1];
  // reductions and scalars
  int32_t wsum[kSelWaves];
  double dred[2 * kSelWaves];
  double saba_u[kMaxGrid];
  double theta;
  int32_t sc[16];
};

enum { kNPool = 0, kBudget, kMono, kBstar, kA, kG, kNX, kXfit, kTotal, kMaxDepth, kNSel, kDepthN };

__device__ __forceinline__ int32_t ptoken(const SelMem &s, int K, int32_t info) {
  return s.cand[(pi_depth(info) - 1) * K + pi_slot(info)];
}

// Is pool entry a ranked before pool entry b?  (score desc, depth asc, token path asc)
__device__ bool pool_before(const SelMem &s, int K, int a, int b) {
  const double sa = s.p_score[a], sb = s.p_score[b];
  if (sa != sb) return sa > sb;
  const int32_t ia = s.p_info[a], ib = s.p_info[b];
  const int da = pi_depth(ia), db = pi_depth(ib);
  if (da != db) return da < db;
  int ta = ptoken(s, K, ia), tb = ptoken(s, K, ib);
  int x = pi_parent(ia), y = pi_parent(ib);
  while (x != y) {
    ta = ptoken(s, K, s.p_info[x]);
    tb = ptoken(s, K, s.p_info[y]);
    x = pi_parent(s.p_info[x]);
    y = pi_parent(s.p_info[y]);
  }
  return ta < tb;
}

// Block-wide exclusive prefix sum of data[0, n) in place; returns the total.
__device__ int block_scan(SelMem &s, int32_t *data, int n) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int per = (n + kSelThreads - 1) / kSelThreads;
  const int lo = tid * per, hi = lo + per < n ? lo + per : n;
  int sum = 0;
  for (int i = lo; i < hi; ++i) sum += data[i];
  int inc = sum;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int v = __shfl_up(inc, o);
    if (lane >= o) inc += v;
  }
  if (lane == kWave - 1) s.wsum[wave] = inc;
  __syncthreads();
  int wbase = 0, total = 0;
  for (int w = 0; w < kSelWaves; ++w) {
    const int v = s.wsum[w];
    if (w < wave) wbase += v;
    total += v;
  }
  int run = wbase + inc - sum;
  for (int i = lo; i < hi; ++i) {
    const int v = data[i];
    data[i] = run;
    run += v;
  }
  __syncthreads();
  return total;
}

// Block-wide min and max of p_score[0, n).
__device__ void block_minmax(SelMem &s, int n, double &mn, double &mx) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  double a = INFINITY, b = -INFINITY;
  for (int i = tid; i < n; i += kSelThreads) {
    const double v = s.p_score[i];
    a = v < a ? v : a;
    b = v > b ? v : b;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double oa = shfl_xor_f64(a, o), ob = shfl_xor_f64(b, o);
    a = oa < a ? oa : a;
    b = ob > b ? ob : b;
  }
  if (lane == 0) {
    s.dred[wave] = a;
    s.dred[kSelWaves + wave] = b;
  }
  __syncthreads();
  mn = s.dred[0];
  mx = s.dred[kSelWaves];
  for (int w = 1; w < kSelWaves; ++w) {
    mn = s.dred[w] < mn ? s.dred[w] : mn;
    mx = s.dred[kSelWaves + w] > mx ? s.dred[kSelWaves + w] : mx;
  }
  __syncthreads();
}

__device__ __forceinline__ int score_bin(double v, double smax, double scale) {
  const double f = (smax - v) * scale;
  int b = static_cast<int>(f);
  return b < kBins - 1 ? (b < 0 ? 0 : b) : kBins - 1;
}

// Keeps the best n_keep entries of the pool (exact), compacts it in pool order
// and sets s.theta to the score of the last kept entry.
__device__ void pool_select(SelMem &s, int K, int n_keep) {
  const int tid = threadIdx.x;
  const int n = s.sc[kNPool];
  double smin, smax;
  block_minmax(s, n, smin, smax);
  const double scale = smax > smin ? static_cast<double>(kBins) / (smax - smin) : 0.0;
  for (int i = tid; i <= kBins; i += kSelThreads) s.hist[i] = 0;
  if (tid == 0) s.sc[kG] = 0;
  __syncthreads();
  for (int i = tid; i < n; i += kSelThreads)
    atomicAdd(&s.hist[score_bin(s.p_score[i], smax, scale)], 1);
  __syncthreads();
  block_scan(s, s.hist, kBins + 1);   // hist[b] = entries in bins < b
  for (int b = tid; b < kBins; b += kSelThreads)
    if (s.hist[b] < n_keep && n_keep <= s.hist[b + 1]) {
      s.sc[kBstar] = b;
      s.sc[kA] = s.hist[b];
    }
  __syncthreads();
  const int bstar = s.sc[kBstar], A = s.sc[kA];
  // boundary bin members, then their exact ranks among themselves
  for (int i = tid; i < n; i += kSelThreads)
    if (score_bin(s.p_score[i], smax, scale) == bstar) s.map[atomicAdd(&s.sc[kG], 1)] = i;
  __syncthreads();
  const int g = s.sc[kG], need = n_keep - A;
  for (int i = tid; i <= n; i += kSelThreads)
    s.aux[i] = i < n && score_bin(s.p_score[i], smax, scale) < bstar;
  __syncthreads();
  for (int j = tid; j < g; j += kSelThreads) {
    const int e = s.map[j];
    int rank = 0;
    for (int q = 0; q < g; ++q) rank += (q != j) && pool_before(s, K, s.map[q], e);
    if (rank < need) s.aux[e] = 1;
    if (rank == need - 1) s.theta = s.p_score[e];
  }
  __syncthreads();
  // stable compaction with parent remapping (parents are always kept)
  double keep_s[kPoolCap / kSelThreads];
  int32_t keep_i[kPoolCap / kSelThreads];
  int keep_to[kPoolCap / kSelThreads];
  block_scan(s, s.aux, n + 1);        // aux[i] = new index if kept; aux[n] = kept count
  int c = 0;
#pragma unroll
  for (int k = 0; k < kPoolCap / kSelThreads; ++k) {
    const int i = tid + k * kSelThreads;
    keep_to[k] = -1;
    if (i < n && s.aux[i + 1] != s.aux[i]) {
      const int32_t info = s.p_info[i];
      const int p = pi_parent(info);
      keep_s[k] = s.p_score[i];
      keep_i[k] = pinfo(p < 0 ? -1 : s.aux[p], pi_depth(info), pi_slot(info), pi_expanded(info));
      keep_to[k] = s.aux[i];
      ++c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kPoolCap / kSelThreads; ++k)
    if (keep_to[k] >= 0) {
      s.p_score[keep_to[k]] = keep_s[k];
      s.p_info[keep_to[k]] = keep_i[k];
    }
  (void)c;
  if (tid == 0) s.sc[kNPool] = n_keep;
  __syncthreads();
}

// Parallel exact top-N for sequences whose edge scores are all <= 0.
__device__ void select_parallel(SelMem &s, const SelectArgs &a, const float *ss,
                                const uint8_t *sc, int n_target) {
  const int tid = threadIdx.x;
  const int L = a.L, K = a.K;
  for (int r = tid; r < K; r += kSelThreads) {
    s.p_score[r] = static_cast<double>(ss[r]);
    s.p_info[r] = pinfo(-1, 1, sc[r], 0);
  }
  if (tid == 0) {
    s.sc[kNPool] = K;
    s.theta = -INFINITY;
  }
  __syncthreads();
  for (;;) {
    if (s.sc[kNPool] > n_target) pool_select(s, K, n_target);
    const int n = s.sc[kNPool];
    // unexpanded prefixes that can still grow
    for (int i = tid; i < n; i += kSelThreads) {
      const int32_t info = s.p_info[i];
      s.aux[i] = !pi_expanded(info) && pi_depth(info) < L;
    }
    __syncthreads();
    const int nx = block_scan(s, s.aux, n);
    if (nx == 0) break;
    for (int i = tid; i < n; i += kSelThreads) {
      const int32_t info = s.p_info[i];
      if (!pi_expanded(info) && pi_depth(info) < L) s.map[s.aux[i]] = i;
    }
    __syncthreads();
    // children of X[j] reaching theta: a prefix of its ranked row; count them
    const double theta = s.theta;
    for (int j = tid; j <= nx; j += kSelThreads) s.aux[j] = 0;
    __syncthreads();
    for (int t = tid; t < nx * K; t += kSelThreads) {
      const int j = t / K, r = t % K;
      const int x = s.map[j];
      const int32_t info = s.p_info[x];
      const int64_t row = (static_cast<int64_t>(pi_depth(info)) * K + pi_slot(info)) * K;
      const bool pass = s.p_score[x] + static_cast<double>(ss[row + r]) >= theta;
      const bool next = r + 1 < K && s.p_score[x] + static_cast<double>(ss[row + r + 1]) >= theta;
      if (pass && !next) s.aux[j] = r + 1;
    }
    __syncthreads();
    // aux[nx] holds the sum; expand the longest prefix of X that fits
    const int total = block_scan(s, s.aux, nx + 1);
    const int room = kPoolCap - n;
    if (tid == 0) s.sc[kXfit] = nx;
    __syncthreads();
    if (total > room)
      for (int j = tid; j < nx; j += kSelThreads)
        if (s.aux[j] <= room && s.aux[j + 1] > room) s.sc[kXfit] = j;
    __syncthreads();
    const int xfit = s.sc[kXfit];
    const int added = s.aux[xfit];
    for (int t = tid; t < xfit * K; t += kSelThreads) {
      const int j = t / K, r = t % K;
      const int cnt = s.aux[j + 1] - s.aux[j];
      if (r >= cnt) continue;
      const int x = s.map[j];
      const int32_t info = s.p_info[x];
      const int d = pi_depth(info);
      const int64_t row = (static_cast<int64_t>(d) * K + pi_slot(info)) * K;
      const int dst = n + s.aux[j] + r;
      s.p_score[dst] = s.p_score[x] + static_cast<double>(ss[row + r]);
      s.p_info[dst] = pinfo(x, d + 1, sc[row + r], 0);
    }
    __syncthreads();
    for (int j = tid; j < xfit; j += kSelThreads) s.p_info[s.map[j]] |= 1 << 25;
    if (tid == 0) s.sc[kNPool] = n + added;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Serial fallback (positive edge scores): lazy best-first with a binary heap.
// Heap entries point at a (parent, rank) stream; popped nodes are written to
// the pool arrays in pop order (parents before children).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int32_t hinfo(int parent, int rank, int slot, int depth) {
  return ((parent + 1) << 18) | (rank << 12) | (slot << 6) | (depth - 1);
}
__device__ __forceinline__ int hi_parent(int32_t v) { return (v >> 18) - 1; }
__device__ __forceinline__ int hi_rank(int32_t v) { return (v >> 12) & 63; }
__device__ __forceinline__ int hi_slot(int32_t v) { return (v >> 6) & 63; }
__device__ __forceinline__ int hi_depth(int32_t v) { return (v & 63) + 1; }

__device__ bool heap_before(const SelMem &s, int K, int a, int b) {
  const double sa = s.h_score[a], sb = s.h_score[b];
  if (sa != sb) return sa > sb;
  const int32_t ia = s.h_info[a], ib = s.h_info[b];
  const int da = hi_depth(ia), db = hi_depth(ib);
  if (da != db) return da < db;
  int ta = s.cand[(da - 1) * K + hi_slot(ia)], tb = s.cand[(db - 1) * K + hi_slot(ib)];
  int x = hi_parent(ia), y = hi_parent(ib);
  while (x != y) {
    ta = ptoken(s, K, s.p_info[x]);
    tb = ptoken(s, K, s.p_info[y]);
    x = pi_parent(s.p_info[x]);
    y = pi_parent(s.p_info[y]);
  }
  return ta < tb;
}

__device__ void heap_swap(SelMem &s, int i, int j) {
  const double sc = s.h_score[i];
  s.h_score[i] = s.h_score[j];
  s.h_score[j] = sc;
  const int32_t in = s.h_info[i];
  s.h_info[i] = s.h_info[j];
  s.h_info[j] = in;
}

__device__ void heap_push(SelMem &s, int K, int &n, double score, int32_t info) {
  int i = n++;
  s.h_score[i] = score;
  s.h_info[i] = info;
  while (i > 0) {
    const int p = (i - 1) >> 1;
    if (!heap_before(s, K, i, p)) break;
    heap_swap(s, i, p);
    i = p;
  }
}

__device__ void heap_pop_root(SelMem &s, int K, int &n) {
  --n;
  if (n == 0) return;
  s.h_score[0] = s.h_score[n];
  s.h_info[0] = s.h_info[n];
  int i = 0;
  for (;;) {
    const int l = 2 * i + 1, r = l + 1;
    int best = i;
    if (l < n && heap_before(s, K, l, best)) best = l;
    if (r < n && heap_before(s, K, r, best)) best = r;
    if (best == i) break;
    heap_swap(s, i, best);
    i = best;
  }
}

__device__ void select_serial(SelMem &s, const SelectArgs &a, const float *ss, const uint8_t *sc,
                              int n_target) {
  const int L = a.L, K = a.K;
  int hn = 0, n_sel = 0;
  if (n_target > 0) heap_push(s, K, hn, static_cast<double>(ss[0]), hinfo(-1, 0, sc[0], 1));
  while (n_sel < n_target && hn > 0) {
    const double score = s.h_score[0];
    const int32_t info = s.h_info[0];
    heap_pop_root(s, K, hn);
    const int p = hi_parent(info), r = hi_rank(info), slot = hi_slot(info), d = hi_depth(info);
    const int i = n_sel++;
    s.p_score[i] = score;
    s.p_info[i] = pinfo(p, d, slot, 1);
    if (r + 1 < K) {   // next sibling under the same parent
      const int pslot = p < 0 ? 0 : pi_slot(s.p_info[p]);
      const double pscore = p < 0 ? 0.0 : s.p_score[p];
      const int64_t off = (static_cast<int64_t>(d - 1) * K + pslot) * K + (r + 1);
      heap_push(s, K, hn, pscore + static_cast<double>(ss[off]), hinfo(p, r + 1, sc[off], d));
    }
    if (d < L) {       // best child of the new node
      const int64_t off = (static_cast<int64_t>(d) * K + slot) * K;
      heap_push(s, K, hn, score + static_cast<double>(ss[off]), hinfo(i, 0, sc[off], d + 1));
    }
  }
  s.sc[kNPool] = n_sel;
}

__global__ void __launch_bounds__(kSelThreads) select_kernel(SelectArgs a, SabaParams sp,
                                                             int use_saba) {
  __shared__ SelMem s;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int L = a.L, K = a.K;
  const float *ss = a.sorted_score + static_cast<int64_t>(b) * L * K * K;
  const uint8_t *sc = a.sorted_child + static_cast<int64_t>(b) * L * K * K;

  // candidates, their rank by token id, and the sign of the edge scores
  for (int i = tid; i < L * K; i += kSelThreads)
    s.cand[i] = a.topk_ids[static_cast<int64_t>(b) * L * K + i];
  if (tid == 0) s.sc[kMono] = 1;
  __syncthreads();
  for (int i = tid; i < L * K; i += kSelThreads) {
    const int l = i / K;
    int r = 0;
    for (int k = 0; k < K; ++k) r += s.cand[l * K + k] < s.cand[i];
    s.idr[i] = static_cast<uint8_t>(r);
  }
  for (int i = tid; i < L * K * K; i += kSelThreads) {
    const int l = i / (K * K), p = (i / K) % K;
    if ((l > 0 || p == 0) && ss[i] > 0.f) s.sc[kMono] = 0;
  }

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
      s.sc[kBudget] = budget;
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

  // ---------------- selection ----------------
  int n_target = s.sc[kBudget] < a.n_max ? s.sc[kBudget] : a.n_max;
  if (n_target < 0) n_target = 0;
  if (s.sc[kMono]) {
    if (n_target > 0) {
      select_parallel(s, a, ss, sc, n_target);
    } else if (tid == 0) {
      s.sc[kNPool] = 0;
    }
  } else if (tid == 0) {
    select_serial(s, a, ss, sc, n_target);
  }
  __syncthreads();
  const int n = s.sc[kNPool];
  if (tid == 0) a.n_nodes[b] = n;

  // ---------------- canonical numbering ----------------
  // Depth by depth: a node's key is (rank of its parent within the parent's
  // depth, rank of its token among that depth's candidates).  Keys are set in
  // a bitmap; a node's rank within its depth is the number of set bits below
  // its key (prefix sum of word popcounts).  aux[i] = rank within depth,
  // map[i] = canonical index.
  if (tid == 0) s.sc[kMaxDepth] = 0;
  __syncthreads();
  for (int i = tid; i < n; i += kSelThreads) atomicMax(&s.sc[kMaxDepth], pi_depth(s.p_info[i]));
  __syncthreads();
  const int max_depth = s.sc[kMaxDepth];
  int offset = 0, n_prev = 1;
  for (int d = 1; d <= max_depth; ++d) {
    const int nwords = (n_prev * K + 31) / 32;
    for (int w = tid; w < nwords; w += kSelThreads) s.hist[w] = 0;
    if (tid == 0) s.sc[kDepthN] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += kSelThreads) {
      const int32_t info = s.p_info[i];
      if (pi_depth(info) != d) continue;
      const int p = pi_parent(info);
      const int key = (p < 0 ? 0 : s.aux[p]) * K + s.idr[(d - 1) * K + pi_slot(info)];
      atomicOr(reinterpret_cast<uint32_t *>(&s.hist[key >> 5]), 1u << (key & 31));
      atomicAdd(&s.sc[kDepthN], 1);
    }
    __syncthreads();
    const int nd = s.sc[kDepthN];
    for (int w = tid; w < nwords; w += kSelThreads)
      s.pcnt[w] = __popc(static_cast<uint32_t>(s.hist[w]));
    __syncthreads();
    block_scan(s, s.pcnt, nwords);
    for (int i = tid; i < n; i += kSelThreads) {
      const int32_t info = s.p_info[i];
      if (pi_depth(info) != d) continue;
      const int p = pi_parent(info);
      const int key = (p < 0 ? 0 : s.aux[p]) * K + s.idr[(d - 1) * K + pi_slot(info)];
      const uint32_t word = static_cast<uint32_t>(s.hist[key >> 5]);
      const int rank = s.pcnt[key >> 5] + __popc(word & ((1u << (key & 31)) - 1u));
      s.aux[i] = rank;          // parents (depth d-1) are not touched here
      s.map[i] = offset + rank;
    }
    __syncthreads();
    offset += nd;
    n_prev = nd;
  }

  // ---------------- emission ----------------
  const int64_t ob = static_cast<int64_t>(b) * a.n_max;
  const int32_t base = a.base_pos[b];
  for (int i = tid; i < a.n_max; i += kSelThreads) {
    if (i < n) {
      const int32_t info = s.p_info[i];
      const int c = s.map[i];
      const int p = pi_parent(info);
      const int cp = p < 0 ? -1 : s.map[p];
      a.tokens[ob + c] = ptoken(s, K, info);
      a.parents[ob + c] = cp;
      a.pos_ids[ob + c] = base + pi_depth(info);
      if (a.node_scores) a.node_scores[ob + c] = s.p_score[i];
      s.hist[c] = cp;           // canonical parents for the mask
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
      if (r < n)
        for (int j = r; j >= 0; j = s.hist[j])
          if ((j >> 6) == wd) bits |= 1ull << (j & 63);
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
