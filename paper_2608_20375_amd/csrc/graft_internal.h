// graft_internal.h -- internal declarations of the HIP library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/graft.h"

namespace graft {

constexpr int kWave = 64;
constexpr int kMaxL = 64;
constexpr int kMaxK = 64;
constexpr int kMaxNodes = 1024;
constexpr int kMaxGrid = 64;
constexpr int kMaxScoreDim = 64;
constexpr int kTdesMaxLossBlocks = 512;
constexpr int kFitSums = 25;        // replay sums: SSE, J^T J (10), J^T r (4), X^T X (6), X^T y (3), y^T y
constexpr int kFitMaxBlocks = 1024;
constexpr int kReadSinkWords = GRAFT_READ_STREAM_SINK_WORDS;

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

// Order-preserving map of an fp32 value to an unsigned key (NaN sorts below -inf
// for the negative-NaN pattern and above +inf otherwise; logits are finite).
__device__ __forceinline__ uint32_t ordered_f32(float x) {
  uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unordered_f32(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}
// Candidate key: larger = earlier in (logit desc, id asc).  0 = empty slot.
__device__ __forceinline__ uint64_t cand_key(float x, uint32_t id) {
  return (static_cast<uint64_t>(ordered_f32(x)) << 32) | static_cast<uint64_t>(~id);
}
__device__ __forceinline__ float cand_value(uint64_t k) {
  return unordered_f32(static_cast<uint32_t>(k >> 32));
}
__device__ __forceinline__ int32_t cand_id(uint64_t k) {
  return static_cast<int32_t>(~static_cast<uint32_t>(k));
}
// Order-preserving map of an fp64 value to an unsigned key.
__device__ __forceinline__ uint64_t ordered_f64(double x) {
  uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  return (u & 0x8000000000000000ull) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double unordered_f64(uint64_t k) {
  const uint64_t u = (k & 0x8000000000000000ull) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
  return __longlong_as_double(static_cast<long long>(u));
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = static_cast<uint32_t>(v), hi = static_cast<uint32_t>(v >> 32);
  lo = __shfl_xor(lo, m);
  hi = __shfl_xor(hi, m);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ double shfl_xor_f64(double v, int m) {
  return __longlong_as_double(static_cast<long long>(
      shfl_xor_u64(static_cast<uint64_t>(__double_as_longlong(v)), m)));
}

// Rank of this lane among the set lanes of `mask` below it.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0));
}

// Value of lane (lane ^ m) for m in {1, 2, 4, 8, 16, 32}.  Masks below 16 use
// DPP lane moves inside a row of 16 (quad_perm for 1 and 2, row_shl/row_shr by
// 4 with a select, row_ror by 8), 16 uses ds_swizzle's xor mode, 32 a permute.
__device__ __forceinline__ uint32_t xor_lane(uint32_t v, int m) {
  const int x = static_cast<int>(v);
  switch (m) {
    case 1: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, true));
    case 2: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, true));
    case 4: {
      const int up = __builtin_amdgcn_mov_dpp(x, 0x104, 0xF, 0xF, true);   // lane + 4
      const int dn = __builtin_amdgcn_mov_dpp(x, 0x114, 0xF, 0xF, true);   // lane - 4
      return static_cast<uint32_t>((__lane_id() & 4) ? dn : up);
    }
    case 8: return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, true));
    case 16: return static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(x, 0x401F));
    default: return static_cast<uint32_t>(__shfl_xor(x, m));
  }
}

__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t v, int m) {
  const uint32_t lo = xor_lane(static_cast<uint32_t>(v), m);
  const uint32_t hi = xor_lane(static_cast<uint32_t>(v >> 32), m);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Inclusive prefix sum over the 64 lanes of a wave: Hillis-Steele steps inside
// rows of 16 lanes (row_shr 1, 2, 4, 8; lanes whose source falls outside the
// row add 0), then row_bcast:15 adds row 0's total to row 1 and row 2's to row
// 3, and row_bcast:31 adds lane 31's value to rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);
  return v;
}
// The same over each half-wave (lanes 0-31 and 32-63) separately.
__device__ __forceinline__ int half_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);
  return v;
}

__device__ __forceinline__ double xor_lane_f64(double v, int m) {
  return __longlong_as_double(static_cast<long long>(
      xor_lane_u64(static_cast<uint64_t>(__double_as_longlong(v)), m)));
}

// Bitonic sort of 64*E keys held by one wave, element index i = e*64 + lane;
// afterwards the keys are in descending order of i.
template <int E>
__device__ __forceinline__ void wave_sort_desc_u32(uint32_t (&k)[E]) {
  const int lane = lane_id();
#pragma unroll
  for (int size = 2; size <= 64 * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= 64) {
        const int es = stride / 64;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((e & es) == 0) {
            const int p = e | es;
            const bool desc = ((e * 64 + lane) & size) == 0;
            const uint32_t a = k[e], b = k[p];
            const bool sw = desc ? (a < b) : (a > b);
            k[e] = sw ? b : a;
            k[p] = sw ? a : b;
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint32_t o = xor_lane(k[e], stride);
          const bool lower = (lane & stride) == 0;
          const bool desc = ((e * 64 + lane) & size) == 0;
          const uint32_t mx = k[e] > o ? k[e] : o, mn = k[e] > o ? o : k[e];
          k[e] = (lower == desc) ? mx : mn;
        }
      }
    }
  }
}

template <int E>
__device__ __forceinline__ void wave_sort_desc(uint64_t (&k)[E]) {
  const int lane = lane_id();
#pragma unroll
  for (int size = 2; size <= 64 * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= 64) {
        const int es = stride / 64;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((e & es) == 0) {
            const int p = e | es;
            const int lo = e * 64 + lane;
            const bool desc = (lo & size) == 0;
            const uint64_t a = k[e], b = k[p];
            const bool sw = desc ? (a < b) : (a > b);
            k[e] = sw ? b : a;
            k[p] = sw ? a : b;
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint64_t o = xor_lane_u64(k[e], stride);
          const int i = e * 64 + lane;
          const bool lower = (lane & stride) == 0;
          const bool desc = (i & size) == 0;
          const uint64_t mx = k[e] > o ? k[e] : o;
          const uint64_t mn = k[e] > o ? o : k[e];
          k[e] = (lower == desc) ? mx : mn;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Context
// ---------------------------------------------------------------------------

struct SabaParams {
  int32_t grid[kMaxGrid];
  int32_t n_grid;
  float phi[4];
  float tau_min, c0, c1, c2;
};

struct ScorerParams {
  float scale, beta;
  int32_t center;
  int32_t score_dim;
  int32_t has_depth_emb;
};

// Per-round intermediates of graft_build_tree, passed from one kernel of the
// round to the next: written by each round before they are read, so nothing
// in them carries over between rounds or needs clearing.
struct RoundScratch {
  int64_t part_slots;      // split-row partials available (rows * splits)
  double *part_stats;      // [part_slots][3]: mL (log2-scaled max), S, T2
  uint64_t *part_keys;     // [part_slots][K]
  int32_t *topk_ids;       // [batch, L, K]
  float *topk_logq;        // [batch, L, K]
  float *row_stats;        // [batch, L, 3]: lse, maxprob, entropy
  float *edge_rows;        // [batch, L, K, K] edge scores: [depth][parent id rank][child id rank]
  int32_t *cand_by_rank;   // [batch, L, K] each depth's candidate tokens in token-id order
  uint8_t *positive;       // [batch, L] 1 if some edge score of that depth is > 0
  float *adj_cos;          // [batch, max(L - 1, 1)] adjacent hidden-state cosines
};

// Byte layout of a RoundScratch for `batch` sequences and part_slots split-row
// partials carved from one buffer at base (every part 256-byte aligned);
// returns the bytes needed.  With base null only the size is computed.
int64_t carve_round_scratch(const graft_dims &d, int batch, int64_t part_slots, char *base,
                            RoundScratch *ws);

}  // namespace graft

struct graft_ctx {
  graft_dims dims;
  int device;
  // per-round intermediates for max_batch sequences, one device allocation
  graft::RoundScratch ws;
  char *ws_base;
  // the library's static scratch array on this context's device
  // (graft_build_tree_static), resolved when the context is created
  char *static_scratch;
  // scorer
  float *proj_parent;      // [V, m]
  float *proj_child;       // [V, m]
  float *depth_emb;        // [L, m] or nullptr
  graft::ScorerParams scorer;
  bool has_scorer;
  bool fuse_edges;         // graft_set_fusion (default on)
  graft::SabaParams saba;
  bool has_saba;
  // history ring
  int32_t *hist_ring;      // [max_batch, window]
  int32_t *hist_pos;       // [max_batch]
  bool has_history;
  // device-side data-error flag
  uint32_t *error_flag;
  // stage timing (graft_profile_begin / graft_profile_end)
  hipEvent_t *prof_build;  // [prof_cap][4]
  hipEvent_t *prof_acc;    // [prof_cap][2]
  int32_t prof_cap, prof_nbuild, prof_nacc;
};

struct graft_tdes {
  graft_tdes_dims dims;
  float *dyc;              // [max_groups K + 2 max_pairs, M16] dL/db of the child-tower rows
  float *dyp;              // [max_groups + 2 max_pairs, M16] dL/da of the parent-tower rows
  float *part_u;           // depth-embedding gradient partials of the loss blocks
  double *part_d;          // [kTdesMaxLossBlocks, 4] scale gradient and objective sums
  float *part_w;           // projection gradient partials of the wgrad blocks
  uint32_t *error_flag;
};

namespace graft {

// Launchers (stream-ordered, no synchronization).  They return hipError_t.
hipError_t launch_logits_pass(graft_ctx *ctx, const RoundScratch &ws, int batch,
                              const uint16_t *logits, const graft_tree_out *out,
                              hipStream_t stream);
hipError_t launch_projection(graft_ctx *ctx, const graft_scorer_desc *d, hipStream_t stream);
hipError_t launch_degen(graft_ctx *ctx, const RoundScratch &ws, int batch,
                        const uint16_t *hidden, int hidden_dim, float *adj_cos_out,
                        hipStream_t stream);
hipError_t launch_edge_scores(graft_ctx *ctx, const RoundScratch &ws, const graft_round_in *in,
                              const graft_tree_out *out, hipStream_t stream);
hipError_t launch_select(graft_ctx *ctx, const RoundScratch &ws, const graft_round_in *in,
                         const graft_tree_out *out, hipStream_t stream);
// True when the selection kernel computes the edge scores and the budget
// itself (the rows fit its LDS stage), so the round launches no edge stage.
bool edges_fused(const graft_ctx *ctx);
hipError_t launch_accept(graft_ctx *ctx, int batch, const int32_t *n_nodes,
                         const int32_t *tokens, const int32_t *parents,
                         const graft_targets *t, int32_t *acc_len, int32_t *acc_nodes,
                         int32_t *bonus, int update_history, hipStream_t stream);
hipError_t launch_set_history(graft_ctx *ctx, int batch, const int32_t *init,
                              hipStream_t stream);
hipError_t launch_mask_to_bias(graft_ctx *ctx, int batch, const int32_t *n_nodes,
                               const uint64_t *mask, void *bias, int dtype, int64_t ld,
                               int64_t batch_stride, hipStream_t stream);
hipError_t launch_commit(graft_ctx *ctx, int batch, const int32_t *acc_len,
                         const int32_t *acc_nodes, const void *src, void *dst, int64_t row_bytes,
                         int n_planes, int64_t sp, int64_t sb, int64_t sr, int64_t dp,
                         int64_t db, int64_t dr, hipStream_t stream);
hipError_t launch_synth_targets(graft_ctx *ctx, int batch, uint64_t seed,
                                const int32_t *root_token, const int32_t *n_nodes,
                                const int32_t *tokens, const int32_t *parents,
                                const int32_t *topk_ids, int32_t *target_root,
                                int32_t *target_node, hipStream_t stream);

// TDES training step: launch sizes for a batch, the instantiated shapes, and
// the three launches (loss_kernel, wgrad_kernel, update_kernel).
struct TdesPlan {
  int loss_blocks, child_blocks, parent_blocks;
};
TdesPlan tdes_plan(const graft_tdes_dims &d, int G, int P);
struct TdesWorkspace {   // element counts of the trainer's buffers
  int64_t dyc, dyp, part_u, part_d, part_w;
};
TdesWorkspace tdes_workspace(const graft_tdes_dims &d);
bool tdes_shape_supported(int E, int m, int L, int K);
hipError_t launch_tdes_step(graft_tdes *t, const float *emb, const graft_tdes_batch *b,
                            const graft_tdes_hyper *h, int32_t step, float *theta, float *m1,
                            float *m2, double *loss, float *grad, hipStream_t stream);

// SABA fit: the replay sums at phi (kFitSums doubles into out, device), with
// the cost's normal equations (with_cost 1) or the residual sum of squares of
// cost c (with_cost 2); partial holds kFitMaxBlocks * kFitSums doubles.
int saba_fit_blocks(int T);
hipError_t launch_replay_sums(int T, int nb, const int32_t *budgets, const float *state,
                              const int32_t *prefix, const float *accepted, const float *latency,
                              const double phi[4], double tau_min, int with_cost,
                              const double c[3], double *partial, double *out, hipStream_t stream);

// Plain read of bytes (a multiple of 16) at src (16-byte aligned); the sink
// holds kReadSinkWords words.
hipError_t launch_read_stream(const void *src, int64_t bytes, uint32_t *sink, hipStream_t stream);

// Number of splits per row used by the logits pass for a given row count.
int logits_splits(const graft_dims &d, int rows);
int logits_part_slots(const graft_dims &d);

}  // namespace graft
