// saba_device.h -- the SABA budget of one sequence, computed by one wave
// (Sec. "State-Aware Budget Allocation"); shared by the edge stage and by the
// selection kernel when it computes the edge scores itself.
#pragma once

#include "graft_internal.h"

namespace graft {

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
// largest U (eq. saba-objective).  Lane 0 stores B_t (and the state when
// asked for it); every lane gets B_t back.
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

__device__ __forceinline__ int saba_budget(const SabaArgs &a, const SabaParams &sp, int b, int L,
                                           const SabaIn &in) {
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
  return budget;
}

// The budget stage's arguments for a round.
inline SabaArgs saba_args(const graft_ctx *ctx, const RoundScratch &ws, const graft_round_in *in,
                          const graft_tree_out *out) {
  SabaArgs sa;
  sa.row_stats = ws.row_stats;
  sa.hist = in->hist;
  sa.hist_ring = ctx->hist_ring;
  sa.prefix_len = in->prefix_len;
  sa.fixed_budget = in->fixed_budget;
  sa.adj_cos = in->hidden ? ws.adj_cos : nullptr;
  sa.window = ctx->dims.hist_window;
  sa.budget = out->budget;
  sa.saba_state = out->saba_state;
  return sa;
}

}  // namespace graft
