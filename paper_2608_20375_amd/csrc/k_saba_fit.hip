// k_saba_fit.hip -- sums over a same-prefix budget-replay log for fitting
// SABA's gain and cost models (the paper's SABA section, eqs. saba-gain and
// saba-cost, fitted on held-out replays as its experimental setup describes).
//
// replay_sums_kernel: one wave per replayed round (lane j = budget j, up to 64
//   budgets), 8 waves per block, rounds strided over the grid.  For the
//   current phi it forms G_j = 1 - exp(-B_j / tau) with tau = max(phi . [1, s],
//   tau_min), the round's best scale A = sum_j a_j G_j / sum_j G_j^2, the
//   residuals r_j = A G_j - a_j and their derivatives by phi at that A (the
//   gradient of the objective with A eliminated), J_jk = -A exp(-B_j / tau)
//   B_j / tau^2 [1, s]_k (0 when tau is clamped), and accumulates the sum of
//   squares, J^T J and J^T r; with the cost flag also X^T X, X^T y and y^T y
//   of the affine cost, X = [1, B, B prefix], or, given a fitted cost, its
//   residual sum of squares.  Lane sums in fp64, then the
//   waves of a block in a fixed order, one partial per block.
// replay_reduce_kernel: one block adds the block partials in a fixed order.
// The Levenberg-Marquardt steps (4 x 4 solves) run on the host.
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kFitWaves = 8;
constexpr int kFitThreads = kFitWaves * kWave;
constexpr int kRedSlices = 32;

struct FitArgs {
  int T, nb;
  const int32_t *budgets;   // device [nb]
  const float *state;       // [T, 3]
  const int32_t *prefix;    // [T]
  const float *accepted;    // [T, nb]
  const float *latency;     // [T, nb]
  double phi0, phi1, phi2, phi3, tau_min;
  double c0, c1, c2;        // with_cost == 2: the fitted cost
  int with_cost;            // 1: normal equations of the cost; 2: its residual sum of squares
  double *partial;          // [blocks, kFitSums]
};

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) v += xor_lane_f64(v, o);
  return v;
}

__global__ void __launch_bounds__(kFitThreads) replay_sums_kernel(FitArgs a) {
  __shared__ double s_w[kFitWaves][kFitSums];
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const bool on = lane < a.nb;
  const double B = on ? static_cast<double>(a.budgets[lane]) : 0.0;
  double acc[kFitSums];
#pragma unroll
  for (int k = 0; k < kFitSums; ++k) acc[k] = 0.0;
  const int W = gridDim.x * kFitWaves;
  for (int t = blockIdx.x * kFitWaves + wave; t < a.T; t += W) {
    const double s1 = a.state[t * 3 + 0], s2 = a.state[t * 3 + 1], s3 = a.state[t * 3 + 2];
    const double pre = static_cast<double>(a.prefix[t]);
    const double av = on ? static_cast<double>(a.accepted[static_cast<int64_t>(t) * a.nb + lane]) : 0.0;
    const double lat = on ? static_cast<double>(a.latency[static_cast<int64_t>(t) * a.nb + lane]) : 0.0;
    const double lin = a.phi0 + a.phi1 * s1 + a.phi2 * s2 + a.phi3 * s3;
    const bool free_tau = lin > a.tau_min;
    const double tau = free_tau ? lin : a.tau_min;
    const double e = on ? exp(-B / tau) : 1.0;
    const double G = 1.0 - e;
    const double sag = wave_sum_f64(av * G), sgg = wave_sum_f64(G * G);
    const double A = sgg > 0.0 ? sag / sgg : 0.0;
    const double r = on ? A * G - av : 0.0;
    // dr/dphi at fixed A
    const double d = (on && free_tau) ? -A * e * B / (tau * tau) : 0.0;
    const double j[4] = {d, d * s1, d * s2, d * s3};
    acc[0] += r * r;
    int k = 1;
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int q = p; q < 4; ++q) acc[k++] += j[p] * j[q];
#pragma unroll
    for (int p = 0; p < 4; ++p) acc[11 + p] += j[p] * r;
    if (a.with_cost == 2 && on) {
      const double rc = a.c0 + a.c1 * B + a.c2 * B * pre - lat;
      acc[24] += rc * rc;
    } else if (a.with_cost == 1 && on) {
      const double x[3] = {1.0, B, B * pre};
      k = 15;
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int q = p; q < 3; ++q) acc[k++] += x[p] * x[q];
#pragma unroll
      for (int p = 0; p < 3; ++p) acc[21 + p] += x[p] * lat;
      acc[24] += lat * lat;
    }
  }
#pragma unroll
  for (int k = 0; k < kFitSums; ++k) {
    const double v = wave_sum_f64(acc[k]);
    if (lane == 0) s_w[wave][k] = v;
  }
  __syncthreads();
  if (tid < kFitSums) {
    double v = 0.0;
    for (int w = 0; w < kFitWaves; ++w) v += s_w[w][tid];
    a.partial[static_cast<int64_t>(blockIdx.x) * kFitSums + tid] = v;
  }
}

// thread (slice, k) adds partials slice, slice + kRedSlices, ... of value k;
// then the slices add in order
__global__ void __launch_bounds__(kRedSlices * 32) replay_reduce_kernel(const double *partial,
                                                                        int blocks, double *out) {
  __shared__ double s_r[kRedSlices][32];
  const int k = threadIdx.x % 32, sl = threadIdx.x / 32;
  double v = 0.0;
  if (k < kFitSums) {
#pragma unroll 8
    for (int b = sl; b < blocks; b += kRedSlices) v += partial[static_cast<int64_t>(b) * kFitSums + k];
  }
  s_r[sl][k] = v;
  __syncthreads();
  if (sl == 0 && k < kFitSums) {
    double t = 0.0;
    for (int s = 0; s < kRedSlices; ++s) t += s_r[s][k];
    out[k] = t;
  }
}

}  // namespace

int saba_fit_blocks(int T) {
  const int b = (T + kFitWaves * 2 - 1) / (kFitWaves * 2);   // about 2 rounds per wave
  return b < 1 ? 1 : (b > kFitMaxBlocks ? kFitMaxBlocks : b);
}

hipError_t launch_replay_sums(int T, int nb, const int32_t *budgets, const float *state,
                              const int32_t *prefix, const float *accepted, const float *latency,
                              const double phi[4], double tau_min, int with_cost,
                              const double c[3], double *partial, double *out, hipStream_t stream) {
  FitArgs a;
  a.T = T;
  a.nb = nb;
  a.budgets = budgets;
  a.state = state;
  a.prefix = prefix;
  a.accepted = accepted;
  a.latency = latency;
  a.phi0 = phi[0];
  a.phi1 = phi[1];
  a.phi2 = phi[2];
  a.phi3 = phi[3];
  a.tau_min = tau_min;
  a.with_cost = with_cost;
  a.c0 = c ? c[0] : 0.0;
  a.c1 = c ? c[1] : 0.0;
  a.c2 = c ? c[2] : 0.0;
  a.partial = partial;
  const int blocks = saba_fit_blocks(T);
  hipLaunchKernelGGL(replay_sums_kernel, dim3(blocks), dim3(kFitThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(replay_reduce_kernel, dim3(1), dim3(kRedSlices * 32), 0, stream, partial, blocks,
                     out);
  return hipGetLastError();
}

}  // namespace graft
