// k_accept.hip -- greedy acceptance walk and the acceptance-history ring.
//
// After the target model has verified a tree it commits the longest accepted
// draft path (the paper's Preliminaries, tree-based speculative decoding; a_t
// in the speculative-decoding paragraph).  Greedy walk: from the root, move to
// the child whose token equals the target's token after the current node; stop
// when no child matches.  A workgroup per sequence stages the tree in LDS with
// one round of loads; one wave then scans it 64 nodes at a time.
// The number of accepted nodes feeds hist_t of the SABA state (mean of the last
// w accepted lengths), kept in a per-sequence device ring.
//
// synth_targets_kernel is a synthetic stand-in for the target model used by
// tests and benchmarks (not part of the method): a counter-based draw keyed on
// each node's identity with splitmix64 (Steele, Lea, Flood, OOPSLA 2014).
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kAccThreads = 256;
static_assert(kMaxNodes % kAccThreads == 0 && kMaxL + 1 <= kAccThreads, "staging slots");

// One workgroup per sequence.  Every thread issues its loads of the tree
// (parents, tokens and, in per-node mode, the targets of all max_nodes slots;
// the padding beyond n_nodes is part of the caller's arrays) before any is
// used, so the walk costs one memory round trip; wave 0 then walks in LDS.
__global__ void __launch_bounds__(kAccThreads)
accept_kernel(int n_max, int L, int window, const int32_t *__restrict__ n_nodes,
              const int32_t *__restrict__ tokens, const int32_t *__restrict__ parents,
              const int32_t *__restrict__ target_root, const int32_t *__restrict__ target_node,
              const int32_t *__restrict__ target_depth, int32_t *__restrict__ acc_len,
              int32_t *__restrict__ acc_nodes, int32_t *__restrict__ bonus,
              int32_t *__restrict__ ring, int32_t *__restrict__ ring_pos, int update) {
  __shared__ int32_t s_par[kMaxNodes], s_tok[kMaxNodes], s_tgt[kMaxNodes + 1];
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = lane_id();
  const int64_t ob = static_cast<int64_t>(b) * n_max;
  const int n_raw = n_nodes[b];
  const int t_root = target_node ? target_root[b] : 0;
  // a fixed number of slots per thread (indices clamped to the arrays), so
  // that all the loads are issued before the first store
  constexpr int kPer = kMaxNodes / kAccThreads;
  int32_t vp[kPer], vt[kPer], vg[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = tid + k * kAccThreads;
    const int64_t ic = ob + (i < n_max ? i : n_max - 1);
    vp[k] = parents[ic];
    vt[k] = tokens[ic];
    vg[k] = target_node ? target_node[ic] : 0;
  }
  // per-depth targets: L + 1 <= kMaxL + 1 entries, one per thread
  const int32_t vd = (!target_node && tid <= L) ? target_depth[static_cast<int64_t>(b) * (L + 1) + tid] : 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int i = tid + k * kAccThreads;
    if (i < n_max) {
      s_par[i] = vp[k];
      s_tok[i] = vt[k];
      if (target_node) s_tgt[i] = vg[k];
    }
  }
  if (!target_node && tid <= L) s_tgt[tid] = vd;
  __syncthreads();
  if (tid >= kWave) return;
  const int n = n_raw < n_max ? (n_raw < 0 ? 0 : n_raw) : n_max;
  int cur = -1, a = 0;
  int t = target_node ? t_root : s_tgt[0];
  // a path has at most L nodes; the bound also ends the walk on malformed
  // trees.  The children of cur are contiguous and follow it in canonical
  // order, so the scan starts after cur.
  while (a < L) {
    int next = -1;
    for (int base = cur + 1; base < n; base += kWave) {
      const int j = base + lane;
      const bool hit = j < n && s_par[j] == cur && s_tok[j] == t;
      const uint64_t m = __ballot(hit);
      if (m) {
        next = base + __builtin_ctzll(m);
        break;
      }
    }
    if (next < 0) break;
    if (lane == 0) acc_nodes[static_cast<int64_t>(b) * L + a] = next;
    ++a;
    cur = next;
    t = target_node ? s_tgt[cur] : s_tgt[a];
  }
  for (int i = a + lane; i < L; i += kWave) acc_nodes[static_cast<int64_t>(b) * L + i] = -1;
  if (lane == 0) {
    acc_len[b] = a;
    bonus[b] = t;
    if (update) {
      const int p = ring_pos[b];
      ring[static_cast<int64_t>(b) * window + p] = a;
      ring_pos[b] = (p + 1) % window;
    }
  }
}

__global__ void set_history_kernel(int total, int window, const int32_t *__restrict__ init,
                                   int32_t *__restrict__ ring, int32_t *__restrict__ pos) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < total) ring[i] = init[i];
  if (i < total / window) pos[i] = 0;
}

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ int32_t synth_target(uint64_t seed, int b, int depth, int32_t ptok, int32_t tok,
                                const int32_t *cand, int L, int K, int64_t V) {
  uint64_t h = splitmix64(seed);
  h = splitmix64(h ^ static_cast<uint64_t>(b));
  h = splitmix64(h ^ static_cast<uint64_t>(depth));
  h = splitmix64(h ^ static_cast<uint64_t>(static_cast<int64_t>(ptok) + 1));
  h = splitmix64(h ^ static_cast<uint64_t>(static_cast<int64_t>(tok) + 1));
  const bool pick = (splitmix64(h ^ 1ull) >> 40) < 13421773ull;
  if (pick && depth < L) {
    const uint64_t h2 = splitmix64(h ^ 2ull);
    int r = h2 ? __builtin_ctzll(h2) : 64;
    if (r > K - 1) r = K - 1;
    return cand[depth * K + r];
  }
  return static_cast<int32_t>(splitmix64(h ^ 3ull) % static_cast<uint64_t>(V));
}

__global__ void __launch_bounds__(256)
synth_targets_kernel(int n_max, int L, int K, int64_t V, uint64_t seed,
                     const int32_t *__restrict__ root_token, const int32_t *__restrict__ n_nodes,
                     const int32_t *__restrict__ tokens, const int32_t *__restrict__ parents,
                     const int32_t *__restrict__ topk_ids, int32_t *__restrict__ target_root,
                     int32_t *__restrict__ target_node) {
  const int b = blockIdx.x;
  const int64_t ob = static_cast<int64_t>(b) * n_max;
  const int32_t *cand = topk_ids + static_cast<int64_t>(b) * L * K;
  const int n = n_nodes[b] < n_max ? n_nodes[b] : n_max;
  const int32_t root = root_token[b];
  if (threadIdx.x == 0) target_root[b] = synth_target(seed, b, 0, -1, root, cand, L, K, V);
  for (int i = threadIdx.x; i < n_max; i += blockDim.x) {
    if (i >= n) {
      target_node[ob + i] = -1;
      continue;
    }
    int depth = 0;
    for (int j = i; j >= 0 && j < n && depth <= L; j = parents[ob + j]) ++depth;
    const int p = parents[ob + i];
    const int32_t ptok = (p < 0 || p >= n) ? root : tokens[ob + p];
    target_node[ob + i] = synth_target(seed, b, depth, ptok, tokens[ob + i], cand, L, K, V);
  }
}

}  // namespace

hipError_t launch_accept(graft_ctx *ctx, int batch, const int32_t *n_nodes,
                         const int32_t *tokens, const int32_t *parents,
                         const graft_targets *t, int32_t *acc_len, int32_t *acc_nodes,
                         int32_t *bonus, int update_history, hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  hipLaunchKernelGGL(accept_kernel, dim3(batch), dim3(kAccThreads), 0, stream, d.max_nodes,
                     d.num_pos, d.hist_window, n_nodes, tokens, parents, t->target_root,
                     t->target_node, t->target_depth, acc_len, acc_nodes, bonus, ctx->hist_ring,
                     ctx->hist_pos, update_history);
  return hipGetLastError();
}

hipError_t launch_set_history(graft_ctx *ctx, int batch, const int32_t *init,
                              hipStream_t stream) {
  const int total = batch * ctx->dims.hist_window;
  hipLaunchKernelGGL(set_history_kernel, dim3((total + 255) / 256), dim3(256), 0, stream, total,
                     ctx->dims.hist_window, init, ctx->hist_ring, ctx->hist_pos);
  return hipGetLastError();
}

hipError_t launch_synth_targets(graft_ctx *ctx, int batch, uint64_t seed,
                                const int32_t *root_token, const int32_t *n_nodes,
                                const int32_t *tokens, const int32_t *parents,
                                const int32_t *topk_ids, int32_t *target_root,
                                int32_t *target_node, hipStream_t stream) {
  const graft_dims &d = ctx->dims;
  hipLaunchKernelGGL(synth_targets_kernel, dim3(batch), dim3(256), 0, stream, d.max_nodes,
                     d.num_pos, d.top_k, static_cast<int64_t>(d.vocab), seed, root_token,
                     n_nodes, tokens, parents, topk_ids, target_root, target_node);
  return hipGetLastError();
}

}  // namespace graft
