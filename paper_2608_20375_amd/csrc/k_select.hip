// k_select.hip -- budgeted best-first selection, canonical emission and the
// ancestor mask; one workgroup per sequence.  The budget B_t comes from the
// edge stage (SABA).
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
//           whose score reaches theta (a parent's edge row is filtered in
//           token-id order; no ranking of the row by score is needed);
//           stop when an expansion adds nothing.
//   A prefix outside the kept set can only gain better competitors, and a
//   skipped child is worse than theta, which only rises, so the result is the
//   exact top N.  Iterations <= depth of the tree + 1.  The pool is
//   append-only: dropped prefixes are marked dead and stay in place (so the
//   children of a prefix always form one contiguous run), and it is compacted
//   only when an expansion would not fit.
//   Otherwise (some positive edge score) one thread runs the heap directly,
//   finding a parent's next child in rank order by a scan of its row.
//
// Emission: canonical numbering (depth ascending, token path ascending), token
//   ids, parent indices, position ids base_pos + depth, path scores, and the
//   ancestor-or-self bitset rows.
//
// Fused edge scores: when a sequence's edge rows fit the LDS stage, the
//   workgroup computes them itself (eqs. tdes-bitower, tdes-center,
//   tdes-score, the edge stage's arithmetic in the same order, so the rows
//   are the same bits) and one of its waves computes the SABA budget; the round
//   then has no separate edge kernel, whose launch and round trips through
//   device memory cost more than the work.
#include <cstddef>

#include "edge_mfma.h"
#include "graft_internal.h"
#include "saba_device.h"

namespace graft {
namespace {

constexpr int kSelThreads = 512;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kPoolCap = 4096;
constexpr int kPerThread = kPoolCap / kSelThreads;
constexpr int kBins = 2048;
constexpr int kStageRows = 4096;   // edge-row floats staged in LDS (all of a sequence's, or its first depths')

// Inputs of the fused edge scores (fused != 0), as the edge stage takes them.
struct EdgeIn {
  int fused;
  int m;                        // score dim, a multiple of 4
  int64_t V;
  uint64_t mdiv4;               // ceil(2^32 / (m / 4)): t / (m / 4) as a multiply-shift
  uint64_t kdiv;                // ceil(2^32 / K)
  const int32_t *topk_ids;      // [B, L, K] candidates, rank order
  const float *topk_logq;       // [B, L, K]
  const int32_t *root_token;    // [B]
  const float *P, *Q;           // [V, m] parent and child projections
  const float *depth_emb;       // [L, m] or nullptr
  ScorerParams sp;
  float *edge_out;              // [B, L, K, K] exported table (rank order) or nullptr
  SabaArgs sa;
  SabaParams saba;
};

struct SelectArgs {
  int L, K, n_max, words;
  const float *edge_rows;       // [B, L, K, K] edge scores, [depth][parent id rank][child id rank]
  const int32_t *cand_by_rank;  // [B, L, K] each depth's candidate tokens in token-id order
  const uint8_t *positive;      // [B, L] some edge score of that depth is > 0
  const int32_t *base_pos;
  const int32_t *budget;        // [B] from the edge stage
  int32_t *n_nodes, *tokens, *parents, *pos_ids;
  uint64_t *mask;
  double *node_scores;
  uint32_t *error_flag;
  EdgeIn e;
};

// Pool entry info: parent + 1 (13 bits) | depth - 1 (6) | rank of the token id
// among its depth's candidates (6) | dead (1).  The edge rows are indexed by
// these ranks (row = parent's rank, column = child's rank).
constexpr uint32_t kDead = 1u << 31;
__device__ __forceinline__ uint32_t pinfo(int parent, int depth, int rank) {
  return static_cast<uint32_t>(parent + 1) | (static_cast<uint32_t>(depth - 1) << 13) |
         (static_cast<uint32_t>(rank) << 19);
}
__device__ __forceinline__ int pi_parent(uint32_t v) { return static_cast<int>(v & 0x1FFF) - 1; }
__device__ __forceinline__ int pi_depth(uint32_t v) { return static_cast<int>((v >> 13) & 63) + 1; }
__device__ __forceinline__ int pi_rank(uint32_t v) { return static_cast<int>((v >> 19) & 63); }
__device__ __forceinline__ bool alive(uint32_t v) { return (v & kDead) == 0; }

struct SelMem {
  double p_score[kPoolCap];
  uint32_t p_info[kPoolCap];
  int32_t map[kPoolCap];
  int32_t aux[kPoolCap + 1];
  int32_t run[kPoolCap];   // run of each entry's children: first index << 8 | length
  union {
    struct {
      alignas(16) int32_t hist[kBins + 1];
      int32_t pcnt[kBins + 1];
    } b;
    struct {                        // serial selector only
      double score[kMaxNodes + 1];
      uint32_t info[kMaxNodes + 1];
    } heap;
  } u;
  int32_t cand[kMaxL * kMaxK];   // candidate tokens of each depth, by token-id rank
  // edge rows of the sequence, staged when they fit
  alignas(16) float rows[kStageRows];
  // reductions and scalars
  int32_t dcnt[kMaxL];   // nodes per depth
  int32_t doff[kMaxL];   // first canonical index of each depth
  int32_t wsum[kSelWaves];
  int32_t first1[kMaxK + 1];   // first child index of each depth-1 entry (first expansion)
  int32_t epos[kSelWaves];     // fused edge scores: some score of the wave's depths is > 0
  double theta;
  unsigned long long thkey;   // ordered key of theta when a whole bin is kept
  unsigned long long lomin;   // ordered key of the smallest score appended
  int32_t sc[16];
};

enum { kNPool = 0, kBudget, kMono, kBstar, kA, kBcnt, kG, kXfit, kMaxDepth, kNSel, kDepthN,
       kMixed, kRootRun, kRHi };

__device__ __forceinline__ int32_t ptoken(const SelMem &s, int K, uint32_t info) {
  return s.cand[(pi_depth(info) - 1) * K + pi_rank(info)];
}

// Is pool entry a ranked before pool entry b?  (score desc, depth asc, token path asc)
__device__ bool pool_before(const SelMem &s, int K, int a, int b) {
  const double sa = s.p_score[a], sb = s.p_score[b];
  if (sa != sb) return sa > sb;
  const uint32_t ia = s.p_info[a], ib = s.p_info[b];
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
  const int inc = wave_incl_scan(sum);
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

constexpr int kBinsPer = kBins / kSelThreads;   // bins per thread in the scan
static_assert(kBins == kBinsPer * kSelThreads && kBinsPer == 4, "4 bins per thread");
static_assert(kBins % (4 * kWave) == 0, "the histogram clears as int4 stores by one wave");
// Histogram slot of a bin: bin 4 t + j of thread t's run is stored at
// j * kSelThreads + t, so the scan's reads (thread t, run position j) hit
// consecutive words.
__device__ __forceinline__ int hslot(int bin) { return ((bin & 3) << 9) | (bin >> 2); }

// The bin holding the n_keep-th entry (bins in descending score order): every
// thread scans its 4 bins and clears them, the waves' totals are combined in
// LDS, and the one thread whose run holds the n_keep-th entry records the bin
// (kBstar), the count before it (kA) and its own count (kBcnt).  Ends with a
// barrier; hist is left cleared.
__device__ __forceinline__ void hist_boundary(SelMem &s, int n_keep) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  int c[kBinsPer], sum = 0;
#pragma unroll
  for (int j = 0; j < kBinsPer; ++j) {
    c[j] = s.u.b.hist[j * kSelThreads + tid];
    sum += c[j];
  }
#pragma unroll
  for (int j = 0; j < kBinsPer; ++j) s.u.b.hist[j * kSelThreads + tid] = 0;
  const int inc = wave_incl_scan(sum);
  if (lane == kWave - 1) s.wsum[wave] = inc;
  __syncthreads();
  // the waves before this one: a fixed-count loop, so that the eight LDS
  // reads are issued together
  int run = inc - sum;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const int v = s.wsum[w];
    run += w < wave ? v : 0;
  }
#pragma unroll
  for (int j = 0; j < kBinsPer; ++j) {
    if (run < n_keep && n_keep <= run + c[j]) {
      s.sc[kBstar] = tid * kBinsPer + j;
      s.sc[kA] = run;
      s.sc[kBcnt] = c[j];
    }
    run += c[j];
  }
  __syncthreads();
}

__device__ __forceinline__ int score_bin(double v, double hi, double scale) {
  const double f = (hi - v) * scale;
  int b = static_cast<int>(f);
  return b < kBins - 1 ? (b < 0 ? 0 : b) : kBins - 1;
}

// Keeps the best n_keep alive entries of pool[0, n) (exact), marks the others
// dead and returns the score of the last kept entry.  Requires more than
// n_keep alive entries, all with scores in [lo, hi], and hist[] cleared (it
// is left cleared).
__device__ double pool_select(SelMem &s, int K, int n, int n_keep, double lo, double hi) {
  const int tid = threadIdx.x;
  const double scale = hi > lo ? static_cast<double>(kBins) / (hi - lo) : 0.0;
  for (int i = tid; i < n; i += kSelThreads) {
    const bool live = alive(s.p_info[i]);
    const int bin = score_bin(s.p_score[i], hi, scale);
    if (live) atomicAdd(&s.u.b.hist[hslot(bin)], 1);
  }
  if (tid == 0) {
    s.sc[kG] = 0;
    s.thkey = ~0ull;
  }
  __syncthreads();
  hist_boundary(s, n_keep);
  // entries past the boundary bin die.  When the whole boundary bin is kept,
  // theta is its smallest score; otherwise its members are listed and ranked.
  const int bstar = s.sc[kBstar], need = n_keep - s.sc[kA];
  const bool whole = s.sc[kBcnt] == need;
  for (int i = tid; i < n; i += kSelThreads) {
    const uint32_t info = s.p_info[i];
    const double v = s.p_score[i];
    const int bin = score_bin(v, hi, scale);
    if (!alive(info)) continue;
    if (bin > bstar) s.p_info[i] = info | kDead;
    else if (bin == bstar) {
      if (whole) atomicMin(&s.thkey, ordered_f64(v));
      else s.map[atomicAdd(&s.sc[kG], 1)] = i;
    }
  }
  __syncthreads();
  if (whole) return unordered_f64(s.thkey);
  // exact ranks inside the boundary bin (only the dead bit of p_info changes
  // here, and the comparisons read the other bits)
  // rank = members with a higher score (independent loads, unrolled) plus,
  // only when some member has the same score, those the full order puts first
  const int g = s.sc[kG];
  for (int j = tid; j < g; j += kSelThreads) {
    const int e = s.map[j];
    const double ve = s.p_score[e];
    int rank = 0, same = 0;
#pragma unroll 8
    for (int q = 0; q < g; ++q) {
      const double vq = s.p_score[s.map[q]];
      rank += vq > ve;
      same += vq == ve;
    }
    if (same > 1) {
      for (int q = 0; q < g; ++q) {
        const int eq = s.map[q];
        rank += (q != j) && s.p_score[eq] == ve && pool_before(s, K, eq, e);
      }
    }
    if (rank >= need) atomicOr(&s.p_info[e], kDead);
    if (rank == need - 1) s.theta = ve;
  }
  __syncthreads();
  return s.theta;
}

// Removes the dead entries of pool[0, n), keeping the order and remapping
// parents (a kept entry's parent is kept).  Returns the new size; *x_lo is
// moved to the new index of the first entry at or after it.
__device__ int pool_compact(SelMem &s, int n, int *x_lo) {
  const int tid = threadIdx.x;
  for (int i = tid; i <= n; i += kSelThreads) s.aux[i] = i < n && alive(s.p_info[i]);
  __syncthreads();
  const int kept = block_scan(s, s.aux, n + 1);   // aux[i] = new index if kept
  double keep_s[kPerThread];
  uint32_t keep_i[kPerThread];
  int32_t keep_r[kPerThread];
  int keep_to[kPerThread];
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int i = tid + k * kSelThreads;
    keep_to[k] = -1;
    if (i < n && s.aux[i + 1] != s.aux[i]) {
      const uint32_t info = s.p_info[i];
      const int p = pi_parent(info);
      keep_s[k] = s.p_score[i];
      keep_i[k] = pinfo(p < 0 ? -1 : s.aux[p], pi_depth(info), pi_rank(info));
      // the run keeps its kept members: aux[j] = new index of the first kept entry >= j
      const int32_t rv = s.run[i];
      const int r0 = rv >> 8, r1 = r0 + (rv & 255);
      keep_r[k] = (s.aux[r0] << 8) | (s.aux[r1] - s.aux[r0]);
      keep_to[k] = s.aux[i];
    }
  }
  int root_run = 0;
  if (threadIdx.x == 0) {
    const int32_t rv = s.sc[kRootRun];
    const int r0 = rv >> 8, r1 = r0 + (rv & 255);
    root_run = (s.aux[r0] << 8) | (s.aux[r1] - s.aux[r0]);
  }
  *x_lo = s.aux[*x_lo];
  __syncthreads();
  if (threadIdx.x == 0) s.sc[kRootRun] = root_run;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k)
    if (keep_to[k] >= 0) {
      s.p_score[keep_to[k]] = keep_s[k];
      s.p_info[keep_to[k]] = keep_i[k];
      s.run[keep_to[k]] = keep_r[k];
    }
  __syncthreads();
  return kept;
}

// Where selection reads the edge rows of a sequence ([depth][parent rank]
// [child rank], rows of K): all of them staged in LDS, or the rows of the
// first depths staged (as many whole depths as the stage holds) and the
// deeper ones read from device memory.
struct LdsRows {
  const float *p;
  __device__ __forceinline__ const float *row(int off) const { return p + off; }
  __device__ __forceinline__ float at(int i) const { return p[i]; }
};
struct SplitRows {
  const float *lds, *glb;
  int split;   // staged floats: [0, split) in LDS, a whole number of depths
  __device__ __forceinline__ const float *row(int off) const {
    return off < split ? lds + off : glb + off;
  }
  __device__ __forceinline__ float at(int i) const { return i < split ? lds[i] : glb[i]; }
};

// Edge-row helpers for K % 4 == 0 with kv = K / 4 groups of four, KV the
// next power of two >= kv.  A row holds the K children's edge scores in
// child-slot order.  Every load is issued unconditionally (clamped to the
// row) before any use, so one memory round trip covers the row.

template <int KV>
__device__ __forceinline__ void load_row(const float *row, int kv, float4 (&v)[KV]) {
  const float4 *r4 = reinterpret_cast<const float4 *>(row);
#pragma unroll
  for (int q = 0; q < KV; ++q) v[q] = r4[q < kv ? q : kv - 1];
}

// Number of children r < K with ps + row[r] >= theta (fp64 sums), and the
// row's smallest edge score.
template <int KV>
__device__ __forceinline__ int count_row(const float4 (&v)[KV], int kv, double ps, double theta,
                                         float &rmin) {
  int c = 0;
  float mn = v[0].x;
#pragma unroll
  for (int q = 0; q < KV; ++q) {
    const int g = (ps + static_cast<double>(v[q].x) >= theta) +
                  (ps + static_cast<double>(v[q].y) >= theta) +
                  (ps + static_cast<double>(v[q].z) >= theta) +
                  (ps + static_cast<double>(v[q].w) >= theta);
    c += q < kv ? g : 0;
    mn = fminf(mn, fminf(fminf(v[q].x, v[q].y), fminf(v[q].z, v[q].w)));   // clamped groups repeat
  }
  rmin = mn;
  return c;
}
template <int KV>
__device__ __forceinline__ int count_reach(const float *row, int kv, double ps, double theta,
                                           float &rmin) {
  float4 v[KV];
  load_row<KV>(row, kv, v);
  return count_row<KV>(v, kv, ps, theta, rmin);
}

// Adds the children of a row that reach theta (scores ps + row[r]) to the
// histogram.
template <int KV>
__device__ __forceinline__ void bin_children(SelMem &s, const float *row, int kv, double theta,
                                             double ps, double hi, double scale) {
  const float4 *r4 = reinterpret_cast<const float4 *>(row);
  float4 v[KV];
#pragma unroll
  for (int q = 0; q < KV; ++q) v[q] = r4[q < kv ? q : kv - 1];
#pragma unroll
  for (int q = 0; q < KV; ++q) {
    const float f[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const double sc = ps + static_cast<double>(f[k]);
      if (q < kv && sc >= theta) atomicAdd(&s.u.b.hist[hslot(score_bin(sc, hi, scale))], 1);
    }
  }
}

// Appends the children of a row that reach theta at dst, dst + 1, ... in
// token-id order (scores ps + row[r], info with parent x at depth d + 1,
// sibling run runv) and returns the smallest appended score.
template <int KV>
__device__ __forceinline__ double append_row(SelMem &s, const float4 (&v)[KV], int kv,
                                             double theta, int dst, int x, int d, double ps,
                                             int32_t runv) {
  double vmin = INFINITY;
#pragma unroll
  for (int q = 0; q < KV; ++q) {
    const float f[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const double sc = ps + static_cast<double>(f[k]);
      const bool take = q < kv && sc >= theta;
      if (take) {
        const int slot = q * 4 + k;
        s.p_score[dst] = sc;
        s.p_info[dst] = pinfo(x, d + 1, slot);
        s.run[dst] = runv;
        vmin = sc < vmin ? sc : vmin;
      }
      dst += take ? 1 : 0;
    }
  }
  return vmin;
}
template <int KV>
__device__ __forceinline__ double append_children(SelMem &s, const float *row, int kv,
                                                  double theta, int dst, int x, int d, double ps,
                                                  int32_t runv) {
  float4 v[KV];
  load_row<KV>(row, kv, v);
  return append_row<KV>(s, v, kv, theta, dst, x, d, ps, runv);
}

// Children of pool entry x (alive, depth < L) that reach theta, and the
// smallest child score (+inf without children).
struct Counted {
  int c;
  double vmin;
};
template <class RS>
__device__ __forceinline__ Counted entry_count(const SelMem &s, const RS &rs, int x, int L,
                                               int K, int kv, int KVP, double theta) {
  const uint32_t info = s.p_info[x];
  const double ps = s.p_score[x];
  if (!alive(info) || pi_depth(info) >= L) return {0, INFINITY};
  const float *row = rs.row((pi_depth(info) * K + pi_rank(info)) * K);
  float rmin = 0.f;
  int c = 0;
  if (KVP == 1) c = count_reach<1>(row, kv, ps, theta, rmin);
  else if (KVP == 2) c = count_reach<2>(row, kv, ps, theta, rmin);
  else if (KVP == 4) c = count_reach<4>(row, kv, ps, theta, rmin);
  else if (KVP == 8) c = count_reach<8>(row, kv, ps, theta, rmin);
  else if (KVP == 16) c = count_reach<16>(row, kv, ps, theta, rmin);
  else {
    rmin = row[0];
    for (int r = 0; r < K; ++r) {
      c += ps + static_cast<double>(row[r]) >= theta;
      rmin = fminf(rmin, row[r]);
    }
  }
  return {c, ps + static_cast<double>(rmin)};
}

// A lower bound of the N-th best score, from a histogram over the alive pool
// entries and the children reaching theta (aux[i] of them) of every entry of
// [x_lo, n): these are all distinct prefixes, so the score at the start of the
// bin that holds the N-th of them bounds the final N-th score from below.
// All the scores lie in [lo, hi]; hist[] is cleared before and after.
template <class RS>
__device__ __forceinline__ double prune_bound(SelMem &s, const RS &rs, int K, int kv, int KVP, int n, int x_lo,
                              int i0, int per, int n_keep, double theta, double lo, double hi) {
  const int tid = threadIdx.x;
  const double scale = hi > lo ? static_cast<double>(kBins) / (hi - lo) : 0.0;
  for (int i = tid; i < n; i += kSelThreads) {
    const bool live = alive(s.p_info[i]);
    const int bin = score_bin(s.p_score[i], hi, scale);
    if (live) atomicAdd(&s.u.b.hist[hslot(bin)], 1);
  }
  const int m = n - x_lo;
  for (int k = 0; k < per; ++k) {
    const int i = i0 + k;
    if (i >= m) break;
    const int c = s.aux[i];
    if (c == 0) continue;
    const int x = x_lo + i;
    const uint32_t info = s.p_info[x];
    const float *row = rs.row((pi_depth(info) * K + pi_rank(info)) * K);
    const double ps = s.p_score[x];
    if (KVP == 1) bin_children<1>(s, row, kv, theta, ps, hi, scale);
    else if (KVP == 2) bin_children<2>(s, row, kv, theta, ps, hi, scale);
    else if (KVP == 4) bin_children<4>(s, row, kv, theta, ps, hi, scale);
    else if (KVP == 8) bin_children<8>(s, row, kv, theta, ps, hi, scale);
    else if (KVP == 16) bin_children<16>(s, row, kv, theta, ps, hi, scale);
    else
      for (int r = 0; r < K; ++r) {
        const double sc = ps + static_cast<double>(row[r]);
        if (sc >= theta) atomicAdd(&s.u.b.hist[hslot(score_bin(sc, hi, scale))], 1);
      }
  }
  __syncthreads();
  hist_boundary(s, n_keep);
  if (scale == 0.0) return -INFINITY;
  // every binned score in bins <= bstar exceeds hi - (bstar + 1) / scale up to
  // rounding, which the margin covers
  const double edge = hi - static_cast<double>(s.sc[kBstar] + 1) / scale;
  return edge - 1e-9 * (fabs(edge) + fabs(hi) + 1.0);
}

// Appends the c children of pool entry x that reach theta at dst (the caller
// counted them), records their sibling run and returns the smallest appended
// score.
template <class RS>
__device__ __forceinline__ double entry_append(SelMem &s, const RS &rs, int x, int K, int kv,
                                               int KVP, double theta, int dst, int c) {
  s.run[x] = (dst << 8) | c;
  const int32_t runv = 0;   // a new entry has no children yet
  const uint32_t info = s.p_info[x];
  const int d = pi_depth(info);
  const float *row = rs.row((d * K + pi_rank(info)) * K);
  const double ps = s.p_score[x];
  if (KVP == 1) return append_children<1>(s, row, kv, theta, dst, x, d, ps, runv);
  if (KVP == 2) return append_children<2>(s, row, kv, theta, dst, x, d, ps, runv);
  if (KVP == 4) return append_children<4>(s, row, kv, theta, dst, x, d, ps, runv);
  if (KVP == 8) return append_children<8>(s, row, kv, theta, dst, x, d, ps, runv);
  if (KVP == 16) return append_children<16>(s, row, kv, theta, dst, x, d, ps, runv);
  double vmin = INFINITY;
  for (int r = 0; r < K; ++r) {
    const double sc = ps + static_cast<double>(row[r]);
    if (sc >= theta) {
      s.p_score[dst] = sc;
      s.p_info[dst] = pinfo(x, d + 1, r);
      s.run[dst] = runv;
      ++dst;
      vmin = sc < vmin ? sc : vmin;
    }
  }
  return vmin;
}

// Cached variants: the caller keeps the entry's row (v) in registers from
// the count to the append.
template <int KV, class RS>
__device__ __forceinline__ Counted entry_count_cached(const SelMem &s, const RS &rs, int x,
                                                      int L, int K, int kv, double theta,
                                                      float4 (&v)[KV]) {
  const uint32_t info = s.p_info[x];
  const double ps = s.p_score[x];
  if (!alive(info) || pi_depth(info) >= L) return {0, INFINITY};
  load_row<KV>(rs.row((pi_depth(info) * K + pi_rank(info)) * K), kv, v);
  float rmin = 0.f;
  const int c = count_row<KV>(v, kv, ps, theta, rmin);
  return {c, ps + static_cast<double>(rmin)};
}
template <int KV>
__device__ __forceinline__ double entry_append_cached(SelMem &s, int x, int K, int kv,
                                                      double theta, int dst, int c,
                                                      const float4 (&v)[KV]) {
  const uint32_t info = s.p_info[x];
  const int d = pi_depth(info);
  s.run[x] = (dst << 8) | c;   // x's children; a new entry has none yet
  return append_row<KV>(s, v, kv, theta, dst, x, d, s.p_score[x], 0);
}

// Smallest of the wave's fp64 values into s.lomin (as an ordered key; +inf is
// neutral): DPP steps inside each row of 16 lanes, then one LDS atomic per row
// (no cross-row lane exchange, whose LDS round trips would serialise).
__device__ __forceinline__ void lomin_update(SelMem &s, double v) {
  uint64_t k = v < INFINITY ? ordered_f64(v) : ~0ull;
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    const uint64_t ok = xor_lane_u64(k, o);
    k = ok < k ? ok : k;
  }
  if ((lane_id() & 15) == 0 && k != ~0ull) atomicMin(&s.lomin, k);
}

// Largest and smallest float of the wave, in every lane: DPP steps inside the
// rows of 16 lanes, then the four row results read as scalars.
__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __uint_as_float(xor_lane(__float_as_uint(v), o)));
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ float wave_min_f32(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fminf(v, __uint_as_float(xor_lane(__float_as_uint(v), o)));
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fminf(fminf(a, b), fminf(c, d));
}

// The parallel selector's starting state, set up by wave 0 while the other
// waves stage the edge rows: the K depth-1 entries in token-id order (r0: the
// depth-1 row, one score per lane, K <= 64), the root's run, lomin at the
// smallest depth-1 score, the largest one in sc[kRHi] (float bits), and a
// cleared histogram.  Harmless when the serial selector runs instead: it
// rewrites the pool from index 0 and uses the union as its heap.
// In two parts for the fused path, whose scratch overlaps the pool until a
// barrier: select_setup_scalars (the histogram, lomin, the root run, the
// largest score) and select_setup_pool (the K entries).
__device__ __forceinline__ void select_setup_pool(SelMem &s, int K, float r0) {
  const int lane = lane_id();
  if (lane < K) {
    s.p_score[lane] = static_cast<double>(r0);
    s.p_info[lane] = pinfo(-1, 1, lane);
    s.run[lane] = 0;
  }
}
__device__ __forceinline__ void select_setup_scalars(SelMem &s, int K, float r0) {
  const int lane = lane_id();
  int4 *h4 = reinterpret_cast<int4 *>(s.u.b.hist);
#pragma unroll
  for (int k = 0; k < kBins / 4 / kWave; ++k) h4[lane + k * kWave] = make_int4(0, 0, 0, 0);
  const float r_hi = wave_max_f32(lane < K ? r0 : -INFINITY);
  const float r_lo = wave_min_f32(lane < K ? r0 : INFINITY);
  if (lane == 0) {
    s.lomin = ordered_f64(static_cast<double>(r_lo));
    s.sc[kRootRun] = K;   // the depth-1 entries: first index 0, K of them
    s.sc[kRHi] = __float_as_int(r_hi);
  }
}
__device__ __forceinline__ void select_setup(SelMem &s, int K, float r0) {
  select_setup_pool(s, K, r0);
  select_setup_scalars(s, K, r0);
}

// Parallel exact top-N for sequences whose edge scores are all <= 0.  Every
// alive unexpanded entry lies in [x_lo, n).  rs: where the edge rows are read
// (LdsRows, SplitRows).
template <class RS, int KVT>
__device__ __forceinline__ int select_parallel(SelMem &s, const SelectArgs &a, const RS &rs,
                               int n_target) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int L = a.L, K = a.K;
  // vector path: K % 4 == 0, kv = K / 4 groups, KVT = next power of two (0:
  // the scalar path)
  const int kv = K / 4;
  constexpr int KVP = KVT;
  // the rows of a thread's first kCache entries stay in registers from the
  // count to the append
  constexpr int kCache = KVT == 0 ? 0 : KVT <= 8 ? 2 : 1;
  constexpr int KVC = KVT > 0 ? KVT : 1;
  float4 cache[kCache > 0 ? kCache : 1][KVC];
  // The depth-1 entries, the cleared histogram, lomin and the root run were
  // set up with the staging (select_setup).  Every prefix scores at most its
  // depth-1 ancestor, so at most the best depth-1 prefix, which is never
  // dropped.
  const double hi = static_cast<double>(__int_as_float(s.sc[kRHi]));
  double theta = -INFINITY;
  bool pruned = false;
  int n = K, n_alive = K, x_lo = 0;
  if (L > 1 && K <= n_target && K + K * K > n_target) {
    // The first expansion keeps every depth-1 prefix and its K * K children
    // all reach theta = -inf, more than N together: bound the N-th score by a
    // histogram of these K + K * K prefixes over [smallest child score, hi]
    // (the bound the prune step below would take after counting them), one
    // (parent rank, child rank) pair per thread.  Depth-1 prefix r scores
    // rs[r] and its row is rs[K * K + r * K ...].
    const int pairs = K * K;
    double pmin = INFINITY;
    for (int j = tid; j < pairs; j += kSelThreads) {
      const double v = static_cast<double>(rs.at(j / K)) + static_cast<double>(rs.at(pairs + j));
      pmin = v < pmin ? v : pmin;
    }
    lomin_update(s, pmin);
    __syncthreads();
    const double lo = unordered_f64(s.lomin);
    const double scale = hi > lo ? static_cast<double>(kBins) / (hi - lo) : 0.0;
    if (tid < K) atomicAdd(&s.u.b.hist[hslot(score_bin(s.p_score[tid], hi, scale))], 1);
    for (int j = tid; j < pairs; j += kSelThreads) {
      const double v = static_cast<double>(rs.at(j / K)) + static_cast<double>(rs.at(pairs + j));
      atomicAdd(&s.u.b.hist[hslot(score_bin(v, hi, scale))], 1);
    }
    __syncthreads();
    hist_boundary(s, n_target);
    if (scale > 0.0) {
      const double edge = hi - static_cast<double>(s.sc[kBstar] + 1) / scale;
      theta = edge - 1e-9 * (fabs(edge) + fabs(hi) + 1.0);
    }
    pruned = true;
  }
  if (L > 1 && K + K * K <= kPoolCap) {
    // The first expansion, of the K depth-1 entries, spread over their K * K
    // (parent, child) pairs (a few per thread) rather than over the K parents.
    // It never takes the prune step (the first bound above is that step; with
    // K + K * K <= N the children are within N; with N < K theta comes from
    // the exact selection here) and always fits in the pool.
    if (n_alive > n_target) {
      theta = pool_select(s, K, n, n_target, unordered_f64(s.lomin), hi);
      n_alive = n_target;
    }
    const int pairs = K * K;   // pair j: child j % K of depth-1 entry j / K, row rs[K * K + j]
    const int pp = (pairs + kSelThreads - 1) / kSelThreads;
    const int j0 = tid * pp < pairs ? tid * pp : pairs;
    const int j1 = j0 + pp < pairs ? j0 + pp : pairs;
    int sum = 0;
    double vmin = INFINITY;
    for (int j = j0; j < j1; ++j) {
      const int r = j / K;
      const double sc = s.p_score[r] + static_cast<double>(rs.at(pairs + j));
      if (alive(s.p_info[r]) && sc >= theta) {
        ++sum;
        vmin = sc < vmin ? sc : vmin;
      }
    }
    const int inc = wave_incl_scan(sum);
    if (lane == kWave - 1) s.wsum[wave] = inc;
    if (theta == -INFINITY) lomin_update(s, vmin);
    __syncthreads();
    int base = 0, added = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const int v = s.wsum[w];
      base += w < wave ? v : 0;
      added += v;
    }
    // this thread's children in pool order from its offset; the owner of an
    // entry's first pair records where the entry's children start
    int dst = K + base + inc - sum;
    for (int j = j0; j < j1; ++j) {
      const int r = j / K, c = j - r * K;
      if (c == 0) s.first1[r] = dst;
      const double sc = s.p_score[r] + static_cast<double>(rs.at(pairs + j));
      if (alive(s.p_info[r]) && sc >= theta) {
        s.p_score[dst] = sc;
        s.p_info[dst] = pinfo(r, 2, c);
        s.run[dst] = 0;
        ++dst;
      }
    }
    if (j0 < j1 && j1 == pairs) s.first1[K] = dst;
    __syncthreads();
    if (tid < K) s.run[tid] = (s.first1[tid] << 8) | (s.first1[tid + 1] - s.first1[tid]);
    n += added;
    n_alive += added;
    x_lo = K;
    pruned = false;
  }
  for (;;) {
    if (n_alive > n_target) {
      // all alive scores are >= theta (or >= the smallest appended score)
      const double lo = theta > -INFINITY ? theta : unordered_f64(s.lomin);
      theta = pool_select(s, K, n, n_target, lo, hi);
      n_alive = n_target;
    }
    // children reaching theta of each entry of [x_lo, n): this thread counts
    // a contiguous run of entries into aux, then a block scan gives offsets
    const int m = n - x_lo;
    const int per = (m + kSelThreads - 1) / kSelThreads;   // <= kPerThread
    const int i0 = tid * per;
    int sum = 0;
    double vmin = INFINITY;
#pragma unroll
    for (int k = 0; k < kCache; ++k) {
      const int i = i0 + k;
      if (k < per && i < m) {
        const Counted e = entry_count_cached<KVC>(s, rs, x_lo + i, L, K, kv, theta, cache[k]);
        s.aux[i] = e.c;
        sum += e.c;
        vmin = e.vmin < vmin ? e.vmin : vmin;
      }
    }
    for (int k = kCache; k < per; ++k) {
      const int i = i0 + k;
      if (i >= m) break;
      const Counted e = entry_count(s, rs, x_lo + i, L, K, kv, KVP, theta);
      s.aux[i] = e.c;
      sum += e.c;
      vmin = e.vmin < vmin ? e.vmin : vmin;
    }
    const int inc = wave_incl_scan(sum);
    if (lane == kWave - 1) s.wsum[wave] = inc;
    if (theta == -INFINITY) lomin_update(s, vmin);
    __syncthreads();
    int base = 0, added = 0;
    for (int w = 0; w < kSelWaves; ++w) {
      const int v = s.wsum[w];
      base += w < wave ? v : 0;
      added += v;
    }
    if (added == 0) break;
    if (!pruned && n_alive + added > n_target && (theta == -INFINITY || n + added > kPoolCap)) {
      // many children: bound the N-th score by a histogram over the pool and
      // the children, then count again against the tighter bound
      const double lo = theta > -INFINITY ? theta : unordered_f64(s.lomin);
      const double bound =
          prune_bound(s, rs, K, kv, KVP, n, x_lo, i0, per, n_target, theta, lo, hi);
      pruned = true;
      if (bound > theta) {
        theta = bound;
        continue;
      }
    }
    pruned = false;
    const bool fit = n + added <= kPoolCap;
    if (!fit && n_alive < n) {
      // the children do not fit: drop the dead entries and count again
      __syncthreads();                                  // wsum is reused
      n = pool_compact(s, n, &x_lo);
      n_alive = n;
      continue;
    }
    int lim = m, dst = n + base + inc - sum;
    if (!fit) {
      // expand the longest run of [x_lo, n) whose children fit; the pool no
      // longer holds one depth per expansion (see canon_levels)
      if (tid == 0) {
        s.aux[m] = 0;
        s.sc[kMixed] = 1;
      }
      __syncthreads();
      block_scan(s, s.aux, m + 1);                      // aux[i] = offset, aux[m] = total
      const int room = kPoolCap - n;
      if (tid == 0) s.sc[kXfit] = m;
      __syncthreads();
      for (int i = tid; i < m; i += kSelThreads)
        if (s.aux[i] <= room && s.aux[i + 1] > room) s.sc[kXfit] = i;
      __syncthreads();
      lim = s.sc[kXfit];
      dst = n + s.aux[i0 < m ? i0 : m];
    }
    const int grown = fit ? added : s.aux[lim];
    if (grown == 0) {               // cannot happen with n_alive <= N_max <= kPoolCap / 4
      if (tid == 0) atomicOr(a.error_flag, 2u);
      break;
    }
    double amin = INFINITY;
#pragma unroll
    for (int k = 0; k < kCache; ++k) {
      const int i = i0 + k;
      if (k < per && i < lim) {
        const int c = fit ? s.aux[i] : s.aux[i + 1] - s.aux[i];
        if (c > 0) {
          const double v = entry_append_cached<KVC>(s, x_lo + i, K, kv, theta, dst, c, cache[k]);
          amin = v < amin ? v : amin;
        }
        dst += c;
      }
    }
    for (int k = kCache; k < per; ++k) {
      const int i = i0 + k;
      if (i >= lim) break;
      const int c = fit ? s.aux[i] : s.aux[i + 1] - s.aux[i];
      if (c > 0) {
        const double v = entry_append(s, rs, x_lo + i, K, kv, KVP, theta, dst, c);
        amin = v < amin ? v : amin;
      }
      dst += c;
    }
    // the smallest appended score (needed only while theta is unset): one LDS
    // atomic per wave
    if (theta == -INFINITY) lomin_update(s, amin);
    __syncthreads();
    n += grown;
    n_alive += grown;
    x_lo += lim;
  }
  if (tid == 0) s.sc[kNSel] = n_alive;
  // cleared scratch for canon_preorder (the caller's barrier publishes it)
  for (int i = tid; i < n; i += kSelThreads) s.aux[i] = 0;
  for (int i = tid; i < kBins; i += kSelThreads) s.u.b.hist[i] = 0;
  for (int i = tid; i < kMaxL; i += kSelThreads) s.dcnt[i] = 0;
  return n;
}

// select_parallel for the row width of K: groups of four (kv = K / 4,
// rounded up to a power of two) or the scalar path when K % 4 != 0.
template <class RS>
__device__ __forceinline__ int select_parallel_k(SelMem &s, const SelectArgs &a, const RS &rs,
                                                 int n_target) {
  const int K = a.K, kv = K / 4;
  if (K & 3) return select_parallel<RS, 0>(s, a, rs, n_target);
  if (kv <= 1) return select_parallel<RS, 1>(s, a, rs, n_target);
  if (kv <= 2) return select_parallel<RS, 2>(s, a, rs, n_target);
  if (kv <= 4) return select_parallel<RS, 4>(s, a, rs, n_target);
  if (kv <= 8) return select_parallel<RS, 8>(s, a, rs, n_target);
  return select_parallel<RS, 16>(s, a, rs, n_target);
}

// Canonical numbering for the parallel selector's pool when every expansion
// appended one whole depth: the depth-1 entries are in token-id order, and an
// expansion walks the previous depth in pool order appending each entry's
// children in token-id order, so by induction the pool holds the depths in
// ascending order, each in canonical (token path) order, dead entries
// interleaved.  The canonical index of an alive entry is then the number of
// alive entries before it: one block-wide count.  Leaves map[i] = canonical
// index.
__device__ void canon_levels(SelMem &s, int n) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int per = (n + kSelThreads - 1) / kSelThreads;   // <= kPerThread
  const int lo = tid * per, hi = lo + per < n ? lo + per : n;
  // the thread's entries' alive bits, every LDS read issued before any is used
  uint32_t bits = 0;
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int i = lo + k < hi ? lo + k : 0;
    const uint32_t info = s.p_info[i];
    bits |= (lo + k < hi && alive(info)) ? 1u << k : 0u;
  }
  const int cnt = __popc(bits);
  const int inc = wave_incl_scan(cnt);
  if (lane == kWave - 1) s.wsum[wave] = inc;
  __syncthreads();
  int run = inc - cnt;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const int v = s.wsum[w];
    run += w < wave ? v : 0;
  }
  for (int k = 0; lo + k < hi; ++k) {
    s.map[lo + k] = run;
    run += (bits >> k) & 1u;
  }
  __syncthreads();
}

// Canonical numbering for the parallel selector's pool, where the children of
// a node occupy one contiguous run (dead entries included).  The canonical
// order is depth ascending, then token path ascending; among nodes of one
// depth the token-path order is the depth-first preorder that visits children
// by increasing token id.  The preorder position of a node is the number of
// its proper ancestors plus, over the node and its ancestors, the sizes of the
// subtrees of their siblings with smaller token ids.  Needs aux[0, n),
// hist[0, kBins) and dcnt[] cleared; leaves map[i] = canonical index.
__device__ void canon_preorder(SelMem &s, int L, int K, int n, int n_sel) {
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  int32_t *bits = s.u.b.hist, *pcnt = s.u.b.pcnt;
  // subtree sizes (aux) and nodes per depth
  for (int i = tid; i < n; i += kSelThreads) {
    const uint32_t info = s.p_info[i];
    if (!alive(info)) continue;
    atomicAdd(&s.dcnt[pi_depth(info) - 1], 1);
    // parents precede their children in the pool
    for (int j = i; j >= 0 && j <= i; j = pi_parent(s.p_info[j])) atomicAdd(&s.aux[j], 1);
  }
  __syncthreads();
  // map[i] = sizes of the subtrees of i's siblings with smaller token ids;
  // the siblings (dead ones included) form i's run
  for (int i = tid; i < n; i += kSelThreads) {
    const uint32_t info = s.p_info[i];
    if (!alive(info)) continue;
    const int p = pi_parent(info), mine = pi_rank(info);
    const int32_t rv = p < 0 ? s.sc[kRootRun] : s.run[p];   // i's siblings
    const int lo = rv >> 8, hi = lo + (rv & 255);
    int left = 0;
    for (int j0 = lo; j0 < hi; j0 += 16) {
      uint32_t o[16];
      int z[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int j = j0 + k < hi ? j0 + k : i;
        o[k] = s.p_info[j];
        z[k] = s.aux[j];
      }
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int sib = static_cast<int>(alive(o[k])) & static_cast<int>(pi_parent(o[k]) == p) &
                        static_cast<int>(pi_rank(o[k]) < mine);
        left += sib ? z[k] : 0;
      }
    }
    s.map[i] = left;
  }
  __syncthreads();
  // preorder positions; one bit per node in its depth's bitmap of positions
  const int W = (n_sel + 31) / 32;                 // <= 32 words per depth
  int pre[kPerThread];
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    const int i = tid + k * kSelThreads;
    pre[k] = -1;
    if (i >= n) continue;
    const uint32_t info = s.p_info[i];
    if (!alive(info)) continue;
    int acc = pi_depth(info) - 1;
    for (int j = i; j >= 0 && j <= i; j = pi_parent(s.p_info[j])) acc += s.map[j];
    pre[k] = acc;
    atomicOr(reinterpret_cast<uint32_t *>(&bits[(pi_depth(info) - 1) * W + (acc >> 5)]),
             1u << (acc & 31));
  }
  __syncthreads();
  // per depth: popcount prefix over its bitmap words (a half-wave per depth),
  // and the first canonical index of each depth (wave 0)
  for (int t = tid; t < L * 32; t += kSelThreads) {
    const int d = t >> 5, w = t & 31;
    const int c = w < W ? __popc(static_cast<uint32_t>(bits[d * W + w])) : 0;
    const int incl = half_incl_scan(c);
    if (w < W) pcnt[d * W + w] = incl - c;
  }
  if (wave == 0) {
    const int c = lane < L ? s.dcnt[lane] : 0;
    const int incl = wave_incl_scan(c);
    if (lane < L) s.doff[lane] = incl - c;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kPerThread; ++k) {
    if (pre[k] < 0) continue;
    const int i = tid + k * kSelThreads;
    const int d0 = pi_depth(s.p_info[i]) - 1, q = pre[k];
    const uint32_t word = static_cast<uint32_t>(bits[d0 * W + (q >> 5)]);
    s.map[i] = s.doff[d0] + pcnt[d0 * W + (q >> 5)] + __popc(word & ((1u << (q & 31)) - 1u));
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Serial fallback (positive edge scores): lazy best-first with a binary heap.
// A heap entry is a (parent, child slot) candidate; popping it pushes the
// parent's next child in rank order and the popped node's best child.  Popped
// nodes are written to the pool arrays in pop order (parents before children).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t hinfo(int parent, int slot, int depth) {
  return (static_cast<uint32_t>(parent + 1) << 18) | (static_cast<uint32_t>(slot) << 6) |
         static_cast<uint32_t>(depth - 1);
}
__device__ __forceinline__ int hi_parent(uint32_t v) { return static_cast<int>(v >> 18) - 1; }
__device__ __forceinline__ int hi_slot(uint32_t v) { return static_cast<int>((v >> 6) & 63); }
__device__ __forceinline__ int hi_depth(uint32_t v) { return static_cast<int>(v & 63) + 1; }

__device__ bool heap_before(const SelMem &s, int K, int a, int b) {
  const double sa = s.u.heap.score[a], sb = s.u.heap.score[b];
  if (sa != sb) return sa > sb;
  const uint32_t ia = s.u.heap.info[a], ib = s.u.heap.info[b];
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
  const double sc = s.u.heap.score[i];
  s.u.heap.score[i] = s.u.heap.score[j];
  s.u.heap.score[j] = sc;
  const uint32_t in = s.u.heap.info[i];
  s.u.heap.info[i] = s.u.heap.info[j];
  s.u.heap.info[j] = in;
}

__device__ void heap_push(SelMem &s, int K, int &n, double score, uint32_t info) {
  int i = n++;
  s.u.heap.score[i] = score;
  s.u.heap.info[i] = info;
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
  s.u.heap.score[0] = s.u.heap.score[n];
  s.u.heap.info[0] = s.u.heap.info[n];
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

// Rank key of child slot c of a row: larger = earlier in (edge score desc,
// token id asc).  Rows are in token-id order, so column c is the id rank.
__device__ __forceinline__ uint64_t child_key(const float *row, int c) {
  return (static_cast<uint64_t>(ordered_f32(row[c] + 0.0f)) << 32) |
         static_cast<uint64_t>(63 - c);
}

// The child of a row that follows key `after` in rank order (~0 for the
// first), by a scan of the row; -1 when none is left.
__device__ __forceinline__ int next_child(const float *row, int K, uint64_t after) {
  uint64_t best = 0ull;
  int slot = -1;
  for (int c = 0; c < K; ++c) {
    const uint64_t k = child_key(row, c);
    if (k < after && k > best) {
      best = k;
      slot = c;
    }
  }
  return slot;
}

__device__ void select_serial(SelMem &s, const SelectArgs &a, const float *rs, int n_target) {
  const int L = a.L, K = a.K;
  int hn = 0, n_sel = 0;
  if (n_target > 0) {
    const int c0 = next_child(rs, K, ~0ull);
    heap_push(s, K, hn, static_cast<double>(rs[c0]), hinfo(-1, c0, 1));
  }
  while (n_sel < n_target && hn > 0) {
    const double score = s.u.heap.score[0];
    const uint32_t info = s.u.heap.info[0];
    heap_pop_root(s, K, hn);
    const int p = hi_parent(info), slot = hi_slot(info), d = hi_depth(info);
    const int i = n_sel++;
    s.p_score[i] = score;
    s.p_info[i] = pinfo(p, d, slot);
    {   // next sibling under the same parent, in rank order
      const int pslot = p < 0 ? 0 : pi_rank(s.p_info[p]);
      const double pscore = p < 0 ? 0.0 : s.p_score[p];
      const float *row = rs + ((d - 1) * K + pslot) * K;
      const int nx = next_child(row, K, child_key(row, slot));
      if (nx >= 0) heap_push(s, K, hn, pscore + static_cast<double>(row[nx]), hinfo(p, nx, d));
    }
    if (d < L) {       // best child of the new node
      const float *row = rs + (d * K + slot) * K;
      const int c0 = next_child(row, K, ~0ull);
      heap_push(s, K, hn, score + static_cast<double>(row[c0]), hinfo(i, c0, d + 1));
    }
  }
  s.sc[kNPool] = n_sel;
  s.sc[kNSel] = n_sel;
}

// Canonical numbering for the serial selector's pool (pop order, no dead
// entries): depth by depth, a node's key is (rank of its parent within the
// parent's depth, rank of its token id).  Keys are set in a bitmap; a node's
// rank within its depth is the number of set bits below its key (prefix sum
// of word popcounts).  aux[i] = rank within depth, map[i] = canonical index.
__device__ void canon_by_depth(SelMem &s, int K, int n) {
  const int tid = threadIdx.x;
  int32_t *bits = s.u.b.hist, *pcnt = s.u.b.pcnt;
  if (tid == 0) s.sc[kMaxDepth] = 0;
  __syncthreads();
  for (int i = tid; i < n; i += kSelThreads) atomicMax(&s.sc[kMaxDepth], pi_depth(s.p_info[i]));
  __syncthreads();
  const int max_depth = s.sc[kMaxDepth];
  int offset = 0, n_prev = 1;
  for (int d = 1; d <= max_depth; ++d) {
    const int nwords = (n_prev * K + 31) / 32;
    for (int w = tid; w < nwords; w += kSelThreads) bits[w] = 0;
    if (tid == 0) s.sc[kDepthN] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += kSelThreads) {
      const uint32_t info = s.p_info[i];
      if (pi_depth(info) != d) continue;
      const int p = pi_parent(info);
      const int key = (p < 0 ? 0 : s.aux[p]) * K + pi_rank(info);
      atomicOr(reinterpret_cast<uint32_t *>(&bits[key >> 5]), 1u << (key & 31));
      atomicAdd(&s.sc[kDepthN], 1);
    }
    __syncthreads();
    const int nd = s.sc[kDepthN];
    for (int w = tid; w < nwords; w += kSelThreads) pcnt[w] = __popc(static_cast<uint32_t>(bits[w]));
    __syncthreads();
    block_scan(s, pcnt, nwords);
    for (int i = tid; i < n; i += kSelThreads) {
      const uint32_t info = s.p_info[i];
      if (pi_depth(info) != d) continue;
      const int p = pi_parent(info);
      const int key = (p < 0 ? 0 : s.aux[p]) * K + pi_rank(info);
      const uint32_t word = static_cast<uint32_t>(bits[key >> 5]);
      const int rank = pcnt[key >> 5] + __popc(word & ((1u << (key & 31)) - 1u));
      s.aux[i] = rank;          // parents (depth d-1) are not touched here
      s.map[i] = offset + rank;
    }
    __syncthreads();
    offset += nd;
    n_prev = nd;
  }
}

// The fused path's scratch, in the pool arrays (p_score .. run), which
// selection first uses after the edge phase: the child rows and the parent
// rows of every depth (L*K rows each of m floats padded to m + 4: 16-byte
// aligned rows that start on different banks), then the candidates' log q
// and ranks by id (L*K each).
constexpr int kFusedScratchFloats = 24576;   // 96 KiB
static_assert(offsetof(SelMem, p_score) == 0 &&
                  kFusedScratchFloats * sizeof(float) <= offsetof(SelMem, u),
              "the fused scratch lies within the pool arrays");
constexpr int kGatherThreads = kSelThreads - kWave;   // waves 0-6 gather, wave 7 budgets
constexpr int kGatherTasks = 10;   // projection loads (16 bytes) in flight per thread

// n / d for n < 2^26 and d <= 64 with mul = ceil(2^32 / d) (exact there:
// the error term n e / (d 2^32), e < d, stays below 1 / d).
__device__ __forceinline__ int fast_div(int n, uint64_t mul) {
  return static_cast<int>((static_cast<uint64_t>(n) * mul) >> 32);
}

// Fused edge scores of sequence b (eqs. tdes-bitower, tdes-center,
// tdes-score), in two phases over the whole workgroup.  First, with no
// barrier between the two round trips: each thread's candidate (tid < L K),
// its log q and its depth's tokens, for its rank by id within the depth
// (selection's row and column order); and every projection row the depths
// need (the child rows g_c + u_d of the K candidates, the parent rows g_p + u_d
// of the previous depth's candidates, or of the root at depth 1), gathered by
// waves 0-6 from token ids read straight from device memory, all loads of a
// batch issued before any store, while wave 7 computes the budget.  Then wave
// w takes depths w, w + 8, ... and forms the scores with the edge stage's
// matrix-core tiles (edge_tiles<MK, NT>, score dim m = 4 MK of 16 or 32, two
// depths interleaved), writing them straight into the LDS rows.  Leaves
// s.rows, s.cand, s.epos, s.sc[kBudget], s.sc[kMixed] and the selector's
// scalars (select_setup_scalars, by wave 0, which scored depth 1); the caller
// writes the depth-1 pool entries after a barrier (the scratch overlaps the
// pool).
template <int MK, int NT>
__device__ __forceinline__ void fused_edges(SelMem &s, const SelectArgs &a, int b) {
  const EdgeIn &e = a.e;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int L = a.L, K = a.K, LK = L * K, m = e.m, m4 = m >> 2, mp4 = m4 + 1;
  const int64_t V = e.V;
  float4 *chd = reinterpret_cast<float4 *>(s.p_score);   // rows (l, c), then parent rows (l, p)
  float4 *par = chd + LK * mp4;
  float *lqr = reinterpret_cast<float *>(par + LK * mp4);
  int32_t *rnk = reinterpret_cast<int32_t *>(lqr + LK);
  const bool saba_wave = wave == kSelWaves - 1;
  SabaIn saba_in{};
  if (saba_wave) saba_in = saba_load(e.sa, e.saba, b, L);
  int32_t root = e.root_token[b];
  if (root < 0 || root >= V) {
    if (tid == 0) atomicOr(a.error_flag, 1u);
    root = 0;
  }
  // Every load first: this thread's candidate (tid < L K <= 512), its log q
  // and the K tokens of its depth (for its rank by id), then the gather tasks'
  // tokens and projection rows, all from device memory, so that no barrier
  // separates the two round trips.
  const int64_t cb = static_cast<int64_t>(b) * LK;
  const int32_t *ids = e.topk_ids + cb;
  const int ci = tid < LK ? tid : 0;
  const int cbase = fast_div(ci, e.kdiv) * K;
  const int32_t ct = ids[ci];
  const float clq = e.topk_logq[cb + ci];
  int4 tv[4 * NT];   // groups past K reread the first and are masked
  if ((K & 3) == 0) {
#pragma unroll
    for (int q = 0; q < 4 * NT; ++q)
      tv[q] = reinterpret_cast<const int4 *>(ids + cbase)[4 * q < K ? q : 0];
  } else {
#pragma unroll
    for (int q = 0; q < 4 * NT; ++q) {
      const int c = 4 * q;
      tv[q] = make_int4(ids[cbase + (c < K ? c : 0)], ids[cbase + (c + 1 < K ? c + 1 : 0)],
                        ids[cbase + (c + 2 < K ? c + 2 : 0)], ids[cbase + (c + 3 < K ? c + 3 : 0)]);
    }
  }
  // the projection rows: 2 L K rows of m4 groups of four, gathered by waves
  // 0-6 while wave 7 computes the budget; ids outside [0, V) (only with
  // non-finite logits) are clamped for the gathers
  const float4 *P4 = reinterpret_cast<const float4 *>(e.P);
  const float4 *Q4 = reinterpret_cast<const float4 *>(e.Q);
  const float4 *U4 = e.sp.has_depth_emb ? reinterpret_cast<const float4 *>(e.depth_emb) : nullptr;
  const int n_tasks = 2 * LK * m4;
  for (int j0 = 0; !saba_wave && j0 < n_tasks; j0 += kGatherTasks * kGatherThreads) {
    int32_t tok[kGatherTasks], dst[kGatherTasks], j4s[kGatherTasks], ls[kGatherTasks];
    bool chd_row[kGatherTasks];
#pragma unroll
    for (int k = 0; k < kGatherTasks; ++k) {
      int j = j0 + k * kGatherThreads + tid;
      j = j < n_tasks ? j : n_tasks - 1;
      const int row = fast_div(j, e.mdiv4);
      j4s[k] = j - row * m4;
      chd_row[k] = row < LK;
      const int rr = chd_row[k] ? row : row - LK;
      ls[k] = fast_div(rr, e.kdiv);
      tok[k] = chd_row[k] ? ids[rr] : (ls[k] == 0 ? root : ids[rr - K]);
      dst[k] = row * mp4 + j4s[k];
    }
    float4 v[kGatherTasks], u[kGatherTasks];
#pragma unroll
    for (int k = 0; k < kGatherTasks; ++k) {
      const int32_t t = (tok[k] < 0 || tok[k] >= V) ? 0 : tok[k];
      v[k] = (chd_row[k] ? Q4 : P4)[static_cast<int64_t>(t) * m4 + j4s[k]];
      u[k] = U4 ? U4[ls[k] * m4 + j4s[k]] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int k = 0; k < kGatherTasks; ++k)
      if (j0 + k * kGatherThreads + tid < n_tasks)
        chd[dst[k]] = make_float4(v[k].x + u[k].x, v[k].y + u[k].y, v[k].z + u[k].z,
                                  v[k].w + u[k].w);
  }
  // ranks by token id within each depth (selection's row and column order)
  if (tid < LK) {
    int r = 0;
#pragma unroll
    for (int q = 0; q < 4 * NT; ++q) {
      const int c = 4 * q;
      r += (c < K && tv[q].x < ct) + (c + 1 < K && tv[q].y < ct) + (c + 2 < K && tv[q].z < ct) +
           (c + 3 < K && tv[q].w < ct);
    }
    rnk[tid] = r;
    lqr[tid] = clq;
    s.cand[cbase + r] = ct;
  }
  if (saba_wave) {
    const int budget = saba_budget(e.sa, e.saba, b, L, saba_in);
    if (lane == 0) s.sc[kBudget] = budget;
  }
  __syncthreads();

  const float fscale = e.sp.scale / sqrtf(static_cast<float>(m));
  const int ld = 4 * mp4;
  // the job of depth l
  auto job_of = [&](int l) {
    const int64_t base = (static_cast<int64_t>(b) * L + l) * K * K;
    return EdgeJob{reinterpret_cast<const float *>(par + l * K * mp4),
                   reinterpret_cast<const float *>(chd + l * K * mp4),
                   l == 0 ? 1 : K,
                   lqr + l * K,
                   rnk + l * K,
                   l == 0 ? nullptr : rnk + (l - 1) * K,
                   s.rows + l * K * K,
                   e.edge_out ? e.edge_out + base : nullptr};
  };
  bool pos = false;
  int l = wave;
  for (; l + kSelWaves < L; l += 2 * kSelWaves) {   // two depths at a time, interleaved
    const EdgeJob jobs[2] = {job_of(l), job_of(l + kSelWaves)};
    pos |= edge_tiles<MK, NT, 2>(jobs, ld, K, fscale, e.sp.beta, e.sp.center);
  }
  if (l < L) {
    const EdgeJob jobs[1] = {job_of(l)};
    pos |= edge_tiles<MK, NT, 1>(jobs, ld, K, fscale, e.sp.beta, e.sp.center);
  }
  if (e.edge_out && wave == 0) {   // depth 1 has one parent row; the others are 0
    const int64_t base = static_cast<int64_t>(b) * L * K * K;
    for (int i2 = K + lane; i2 < K * K; i2 += kWave) e.edge_out[base + i2] = 0.f;
  }
  const bool any_pos = __ballot(pos) != 0ull;
  if (lane == 0) s.epos[wave] = any_pos ? 1 : 0;
  if (tid == 0) s.sc[kMixed] = 0;
  if (wave == 0) {
    // wave 0 scored depth 1: the selector's scalars now, its pool entries
    // after the barrier
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    select_setup_scalars(s, K, lane < K ? s.rows[lane] : 0.f);
  }
}

// The inputs the edge stage left in device memory for sequence b: wave 0
// reads the budget and the sign flags and sets up the parallel selector from
// the depth-1 row; waves 1.. stage the edge rows (16-byte loads, all issued
// before the stores): all of them when they fit, else those of the first
// depths (n_stage floats, as many whole depths as the stage holds).
__device__ __forceinline__ void load_edge_stage(SelMem &s, const SelectArgs &a, int b,
                                                const float *ss, int n_stage) {
  const int tid = threadIdx.x;
  const int L = a.L, K = a.K;
  int budget0 = 0;
  bool pos0 = false;
  float r0 = 0.f;   // the depth-1 row, one score per lane
  if (tid < kWave) {
    budget0 = a.budget[b];
    pos0 = tid < L && a.positive[static_cast<int64_t>(b) * L + tid] != 0;
    r0 = ss[tid < K ? tid : 0];
  }
  // each depth's candidate tokens in token-id order (written by the edge stage)
  for (int i = tid; i < L * K; i += kSelThreads)
    s.cand[i] = a.cand_by_rank[static_cast<int64_t>(b) * L * K + i];
  constexpr int kStageThreads = kSelThreads - kWave;
  if (tid >= kWave && ((L * K * K) % 4 != 0 || n_stage % 4 != 0)) {
    for (int i = tid - kWave; i < n_stage; i += kStageThreads) s.rows[i] = ss[i];
  } else if (tid >= kWave) {
    // L*K*K is a multiple of 4 here, so the sequence's base is 16-byte aligned
    constexpr int kF4 = (kStageRows / 4 + kStageThreads - 1) / kStageThreads;
    const int t = tid - kWave;
    const int nf4 = n_stage / 4;
    const float4 *src_f = reinterpret_cast<const float4 *>(ss);
    float4 vf[kF4];
#pragma unroll
    for (int k = 0; k < kF4; ++k) {
      const int i = t + k * kStageThreads;
      vf[k] = src_f[i < nf4 ? i : nf4 - 1];
    }
#pragma unroll
    for (int k = 0; k < kF4; ++k)
      if (t + k * kStageThreads < nf4) reinterpret_cast<float4 *>(s.rows)[t + k * kStageThreads] = vf[k];
  }
  // wave 0: the budget, the sign flags and the selector's starting state
  if (tid < kWave) {
    select_setup(s, K, r0);
    const bool mono = __ballot(pos0) == 0ull;
    if (tid == 0) {
      s.sc[kBudget] = budget0;
      s.sc[kMono] = mono ? 1 : 0;
      s.sc[kMixed] = 0;
    }
  }
}

// FUSED: the edge scores and the budget are computed here (a.e), else read
// from the edge stage; two instantiations, so that the unfused kernel carries
// none of the fused code.
template <bool FUSED>
__global__ void __launch_bounds__(kSelThreads) select_kernel(SelectArgs a) {
  __shared__ SelMem s;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int L = a.L, K = a.K;
  const float *ss = a.edge_rows + static_cast<int64_t>(b) * L * K * K;

  constexpr bool fused = FUSED;
  const int n_stage = (L * K * K <= kStageRows ? L : kStageRows / (K * K)) * K * K;
  const bool staged = fused || n_stage == L * K * K;   // the fused path stages every row
  if constexpr (fused) {
    // the edge stage's tile shapes: m = 4 MK in {16, 32}, NT column tiles of 16
    if (a.e.m == 16) {
      if (K <= 16) fused_edges<4, 1>(s, a, b);
      else if (K <= 32) fused_edges<4, 2>(s, a, b);
      else fused_edges<4, 4>(s, a, b);
    } else {
      if (K <= 16) fused_edges<8, 1>(s, a, b);
      else if (K <= 32) fused_edges<8, 2>(s, a, b);
      else fused_edges<8, 4>(s, a, b);
    }
    __syncthreads();   // the scratch overlaps the pool the setup writes
    if (tid < kWave) select_setup_pool(s, K, tid < K ? s.rows[tid] : 0.f);
  } else {
    load_edge_stage(s, a, b, ss, n_stage);
  }
  __syncthreads();

  // ---------------- selection ----------------
  int n_target = s.sc[kBudget] < a.n_max ? s.sc[kBudget] : a.n_max;
  if (n_target < 0) n_target = 0;
  bool mono;
  if constexpr (fused) {
    int any = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) any |= s.epos[w];
    mono = any == 0;
  } else {
    mono = s.sc[kMono] != 0;
  }
  if (mono) {
    if (n_target > 0) {
      const int n_pool = staged ? select_parallel_k(s, a, LdsRows{s.rows}, n_target)
                                : select_parallel_k(s, a, SplitRows{s.rows, ss, n_stage},
                                                    n_target);
      if (tid == 0) s.sc[kNPool] = n_pool;
    } else if (tid == 0) {
      s.sc[kNPool] = 0;
      s.sc[kNSel] = 0;
    }
  } else if (tid == 0) {
    if (staged) select_serial(s, a, s.rows, n_target);
    else select_serial(s, a, ss, n_target);
  }
  __syncthreads();
  const int n = s.sc[kNPool];       // pool entries, dead ones included
  const int n_sel = s.sc[kNSel];    // selected nodes
  if (tid == 0) a.n_nodes[b] = n_sel;

  // ---------------- canonical numbering ----------------
  if (mono && s.sc[kMixed] == 0) canon_levels(s, n);
  else if (mono) canon_preorder(s, L, K, n, n_sel);
  else canon_by_depth(s, K, n);

  // ---------------- emission ----------------
  const int64_t ob = static_cast<int64_t>(b) * a.n_max;
  const int32_t base = a.base_pos[b];
  int32_t *cpar = s.u.b.hist;       // canonical parents, for the mask
  int32_t *gpar = s.u.b.pcnt;       // canonical grandparents
  for (int i = tid; i < n; i += kSelThreads) {
    const uint32_t info = s.p_info[i];
    if (!alive(info)) continue;
    const int c = s.map[i];
    const int p = pi_parent(info);
    const int cp = p < 0 ? -1 : s.map[p];
    const int pp = p < 0 ? -1 : pi_parent(s.p_info[p]);
    a.tokens[ob + c] = ptoken(s, K, info);
    a.parents[ob + c] = cp;
    a.pos_ids[ob + c] = base + pi_depth(info);
    if (a.node_scores) a.node_scores[ob + c] = s.p_score[i];
    cpar[c] = cp;
    gpar[c] = pp < 0 ? -1 : s.map[pp];
  }
  for (int c = n_sel + tid; c < a.n_max; c += kSelThreads) {
    a.tokens[ob + c] = -1;
    a.parents[ob + c] = -1;
    a.pos_ids[ob + c] = -1;
    if (a.node_scores) a.node_scores[ob + c] = 0.0;
  }
  __syncthreads();

  // ---------------- ancestor mask ----------------
  // Each wave takes 64 rows at a time, one per lane: a single walk up the
  // canonical parents (which precede their children, so the indices
  // decrease), two levels per LDS round trip (parent and grandparent read
  // together), emits the row's words from the highest down into LDS (rows
  // padded by one word against bank conflicts); the wave then copies the 64
  // rows out with consecutive lanes on consecutive words.  The pool arrays
  // are free by now and hold the staging rows.
  if (a.mask) {
    const int words = a.words, pitch = words + 1;
    const int lane = lane_id(), wave = tid / kWave;
    const uint32_t recip = (65536u + words - 1) / words;   // t / words for t < 64 * 16
    uint64_t *stage = reinterpret_cast<uint64_t *>(s.p_score) + wave * kWave * pitch;
    uint64_t *mseq = a.mask + static_cast<int64_t>(b) * a.n_max * words;
    for (int base = wave * kWave; base < a.n_max; base += kSelThreads) {
      const int r = base + lane;
      uint64_t *my = stage + lane * pitch;
      int w = words - 1;
      if (r < n_sel) {
        for (; w > (r >> 6); --w) my[w] = 0ull;
        uint64_t bits = 1ull << (r & 63);
        for (int j = r;;) {
          const int p1 = cpar[j], p2 = gpar[j];
          if (p1 < 0 || p1 >= j) break;
          for (; (p1 >> 6) < w; --w) {
            my[w] = bits;
            bits = 0;
          }
          bits |= 1ull << (p1 & 63);
          if (p2 < 0 || p2 >= p1) break;
          for (; (p2 >> 6) < w; --w) {
            my[w] = bits;
            bits = 0;
          }
          bits |= 1ull << (p2 & 63);
          j = p2;
        }
        my[w--] = bits;
      }
      for (; w >= 0; --w) my[w] = 0ull;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int rows = a.n_max - base < kWave ? a.n_max - base : kWave;
      for (int t = lane; t < rows * words; t += kWave) {
        const int rr = static_cast<int>((static_cast<uint32_t>(t) * recip) >> 16);
        mseq[static_cast<int64_t>(base) * words + t] = stage[t + rr];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
}

}  // namespace

bool edges_fused(const graft_ctx *ctx) {
  const graft_dims &d = ctx->dims;
  const int L = d.num_pos, K = d.top_k, m = ctx->scorer.score_dim;
  return ctx->fuse_edges && (m == 16 || m == 32) && L * K * K <= kStageRows &&
         L * K <= kSelThreads && 2 * L * K * (m + 4) + 2 * L * K <= kFusedScratchFloats;
}

hipError_t launch_select(graft_ctx *ctx, const RoundScratch &ws, const graft_round_in *in,
                         const graft_tree_out *out, hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  SelectArgs a;
  a.L = d.num_pos;
  a.K = d.top_k;
  a.n_max = d.max_nodes;
  a.words = (d.max_nodes + 63) / 64;
  a.edge_rows = ws.edge_rows;
  a.cand_by_rank = ws.cand_by_rank;
  a.positive = ws.positive;
  a.base_pos = in->base_pos;
  a.budget = out->budget;
  a.n_nodes = out->n_nodes;
  a.tokens = out->tokens;
  a.parents = out->parents;
  a.pos_ids = out->pos_ids;
  a.mask = out->mask;
  a.node_scores = out->node_scores;
  a.error_flag = ctx->error_flag;
  EdgeIn &e = a.e;
  e = EdgeIn{};
  e.fused = edges_fused(ctx) ? 1 : 0;
  if (e.fused) {
    const int m = ctx->scorer.score_dim, m4 = m / 4;
    e.m = m;
    e.V = d.vocab;
    e.mdiv4 = ((1ull << 32) + static_cast<uint64_t>(m4) - 1) / static_cast<uint64_t>(m4);
    e.kdiv = ((1ull << 32) + static_cast<uint64_t>(d.top_k) - 1) / static_cast<uint64_t>(d.top_k);
    e.topk_ids = ws.topk_ids;
    e.topk_logq = ws.topk_logq;
    e.root_token = in->root_token;
    e.P = ctx->proj_parent;
    e.Q = ctx->proj_child;
    e.depth_emb = ctx->depth_emb;
    e.sp = ctx->scorer;
    e.edge_out = out->edge_scores;
    e.sa = saba_args(ctx, ws, in, out);
    e.saba = ctx->saba;
  }
  if (e.fused)
    hipLaunchKernelGGL(select_kernel<true>, dim3(in->batch), dim3(kSelThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(select_kernel<false>, dim3(in->batch), dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace graft
