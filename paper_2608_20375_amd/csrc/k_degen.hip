// k_degen.hip -- representation degeneration of the SABA decoding state (Sec.
// "State-Aware Budget Allocation", degen_t): the cosine similarity
//   r_d = <h_d, h_{d+1}> / (|h_d| |h_{d+1}|)
// of the drafter's hidden states at adjacent draft positions d, d + 1 of a
// sequence (0 when either state is the zero vector).  The budget stage turns
// them into degen = mean_d r_d + (r_{L-1} - r_1).
//
// degen_kernel: one workgroup per (sequence, run of up to kPairs adjacent
// pairs).  It reads the kPairs + 1 hidden rows of its run once, 16 bytes a
// load, every load of a lane issued before any arithmetic; each lane keeps
// fp32 partial sums of the rows' squared norms and of the adjacent products
// over the vectors it owns; the partials are summed in fp64 across the wave
// (DPP) and across the waves (LDS).  HBM-bound: each row is read once, plus
// one shared row between neighbouring runs.
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kDegenThreads = 256;
constexpr int kDegenWaves = kDegenThreads / kWave;
constexpr int kPairs = 4;                 // adjacent pairs per workgroup
constexpr int kRows = kPairs + 1;
constexpr int kVecPerLane = 2;            // 16-byte vectors per row per lane per step
constexpr int kAcc = kRows + kPairs;      // norms, then adjacent products

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void bf16x8(const u32x4 q, float (&v)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(q[i] << 16);
    v[2 * i + 1] = __uint_as_float(q[i] & 0xFFFF0000u);
  }
}

__global__ void __launch_bounds__(kDegenThreads)
degen_kernel(const uint16_t *__restrict__ hidden, int L, int H, int runs,
             float *__restrict__ adj_cos, float *__restrict__ adj_cos_out) {
  __shared__ double s_part[kDegenWaves][kAcc];
  const int b = blockIdx.x / runs;
  const int d0 = (blockIdx.x % runs) * kPairs;
  const int np = (L - 1 - d0) < kPairs ? (L - 1 - d0) : kPairs;   // pairs of this run, >= 1
  const int nr = np + 1;                                          // rows of this run
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int64_t nv = H / 8;                                       // vectors per row
  const u32x4 *base =
      reinterpret_cast<const u32x4 *>(hidden + (static_cast<int64_t>(b) * L + d0) * H);

  float acc[kAcc];
#pragma unroll
  for (int a = 0; a < kAcc; ++a) acc[a] = 0.f;
  for (int64_t v0 = 0; v0 < nv; v0 += kVecPerLane * kDegenThreads) {
    u32x4 q[kVecPerLane][kRows];
#pragma unroll
    for (int u = 0; u < kVecPerLane; ++u) {
      const int64_t v = v0 + u * kDegenThreads + tid;
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        q[u][r] = u32x4{0u, 0u, 0u, 0u};
        if (r < nr && v < nv) q[u][r] = __builtin_nontemporal_load(base + r * nv + v);
      }
    }
#pragma unroll
    for (int u = 0; u < kVecPerLane; ++u) {
      float x[kRows][8];
#pragma unroll
      for (int r = 0; r < kRows; ++r) bf16x8(q[u][r], x[r]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
#pragma unroll
        for (int r = 0; r < kRows; ++r) acc[r] = __builtin_fmaf(x[r][e], x[r][e], acc[r]);
#pragma unroll
        for (int p = 0; p < kPairs; ++p)
          acc[kRows + p] = __builtin_fmaf(x[p][e], x[p + 1][e], acc[kRows + p]);
      }
    }
  }
  // rows past the run were loaded as zeros, so their sums are 0
#pragma unroll
  for (int a = 0; a < kAcc; ++a) {
    double s = static_cast<double>(acc[a]);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) s += xor_lane_f64(s, o);
    if (lane == 0) s_part[wave][a] = s;
  }
  __syncthreads();
  if (tid < np) {
    double nn[2] = {0.0, 0.0}, dot = 0.0;
#pragma unroll
    for (int w = 0; w < kDegenWaves; ++w) {
      nn[0] += s_part[w][tid];
      nn[1] += s_part[w][tid + 1];
      dot += s_part[w][kRows + tid];
    }
    const double r = (nn[0] > 0.0 && nn[1] > 0.0) ? dot / sqrt(nn[0] * nn[1]) : 0.0;
    const int64_t o = static_cast<int64_t>(b) * (L - 1) + d0 + tid;
    adj_cos[o] = static_cast<float>(r);
    if (adj_cos_out) adj_cos_out[o] = static_cast<float>(r);
  }
}

}  // namespace

hipError_t launch_degen(graft_ctx *ctx, const RoundScratch &ws, int batch,
                        const uint16_t *hidden, int hidden_dim, float *adj_cos_out,
                        hipStream_t stream) {
  const int L = ctx->dims.num_pos;
  if (L < 2) return hipSuccess;
  const int runs = (L - 1 + kPairs - 1) / kPairs;
  hipLaunchKernelGGL(degen_kernel, dim3(static_cast<unsigned>(batch * runs)),
                     dim3(kDegenThreads), 0, stream, hidden, L, hidden_dim, runs, ws.adj_cos,
                     adj_cos_out);
  return hipGetLastError();
}

}  // namespace graft
