// k_tdes_train.hip -- one training step of the TDES edge scorer (the paper's
// Target-Distilled Edge Scoring section: scorer eq. tdes-bitower; objectives
// KL, pairwise margin and class-balanced BCE, summed by eq. tdes-training;
// AdamW as in the training setup of the experiments).
//
// train_kernel: every wave takes a contiguous share of the work items, weighted
//   by cost (a group of K children costs 1, a tile of 8 pairs 2).  For a group
//   it gathers the K child embedding rows with 16-byte loads, projects them
//   through g_child with MFMA (v_mfma_f32_16x16x4_f32: 16 rows x 16 score
//   dimensions per instruction, g_child staged in LDS), projects the parent
//   row through g_parent on the VALU, then forms f, both softmaxes over the
//   children, the KL and BCE terms and dL/df in registers.  The weight
//   gradient e^T dY is one more MFMA contraction over the rows, accumulated
//   in per-wave fp32 registers; its embedding operand is re-read (from L1/L2)
//   in the transposed lane layout the contraction needs.  The rank-1 updates
//   of four groups' parents share one contraction step.  A pair tile projects
//   16 parent rows and 16 child rows the same way.  At the end the block sums
//   its waves' accumulators in a fixed order and writes one partial gradient.
// update_kernel: sums the block partials in fp64 in block order (so a step is
//   deterministic), then applies AdamW to every parameter.
//
// The projections are dense contractions (rows x E x m), so they run on the
// matrix cores; fp32 MFMA has twice the fp32 VALU rate here.
#include <cmath>

#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kTrainWaves = 8;
constexpr int kTrainThreads = kTrainWaves * kWave;
constexpr int kMaxEM = 4096;          // E * ceil(m / 16) * 16
constexpr int kMaxLM = 1024;          // L * ceil(m / 16) * 16
constexpr int kMaxSG = 68;            // LDS row stride of a staged projection
constexpr int kMaxGs = 4608;          // max E * (M16 + 4) over supported shapes

typedef float v4f __attribute__((ext_vector_type(4)));

struct TrainArgs {
  const float *emb;      // [V, E]
  const float *theta;    // [gp E*m | gc E*m | u L*m | s]
  int V, E, m, L, K;
  int G, P;
  const int32_t *parent, *depth, *child, *target, *pairs;
  const float *logq, *z;
  float c_kl, c_bce, c_pair, gamma, w1;
  float *part_g;         // [blocks, 2*E*m + L*m]
  double *part_d;        // [blocks, 4]: ds, sum KL, sum pair, sum BCE
  uint32_t *error_flag;
};

__device__ __forceinline__ float xorf(float v, int m) {
  return __uint_as_float(xor_lane(__float_as_uint(v), m));
}
// sum over the 16 lanes of a row (lanes with equal lane / 16)
__device__ __forceinline__ float sum16(float v) {
  v += xorf(v, 1);
  v += xorf(v, 2);
  v += xorf(v, 4);
  v += xorf(v, 8);
  return v;
}
// sum / max over the 4 rows of 16 lanes (lanes with equal lane % 16)
__device__ __forceinline__ float sum_rows(float v) {
  v += xorf(v, 16);
  v += xorf(v, 32);
  return v;
}
__device__ __forceinline__ float max_rows(float v) {
  v = fmaxf(v, xorf(v, 16));
  v = fmaxf(v, xorf(v, 32));
  return v;
}
__device__ __forceinline__ double sum_rows_f64(double v) {
  v += xor_lane_f64(v, 16);
  v += xor_lane_f64(v, 32);
  return v;
}
// log(1 + e^x) without overflow
__device__ __forceinline__ float softplus(float x) {
  return fmaxf(x, 0.0f) + log1pf(expf(-fabsf(x)));
}
__device__ __forceinline__ float sigmoid(float x) {
  const float e = expf(-fabsf(x));
  return x >= 0.0f ? 1.0f / (1.0f + e) : e / (1.0f + e);
}
__device__ __forceinline__ v4f mfma(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
// Orders this wave's LDS accesses (a wave's DS instructions complete in order).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct alignas(16) WaveScratch {
  float delta[kMaxK];      // dL/df of a group's rows
  float f[kMaxK];          // f of a group's rows
  float dot[kMaxK];        // (g_p + u).(g_c + u) / sqrt(m) of a group's rows
  float xv[128];           // an E-vector
  float pend[4][kMaxScoreDim];  // dA of up to four groups awaiting their parents' update
  int32_t ptok[4];              // their parent tokens
  int32_t tok[kMaxK];      // a group's child tokens; a pair tile's parent tokens
  int32_t tok2[16];        // a pair tile's child tokens
  int32_t dep[16];         // a pair tile's depths
  float tile[16 * kMaxSG]; // dY of a pair tile, transposed through LDS
};

struct TrainLds {
  float gs[2][kMaxGs];                    // g_parent, g_child [E][SG]; later the block sums
  float us[kMaxLM];                       // u [L][M16]
  float du[kTrainWaves][kMaxLM];          // per-wave depth-embedding gradients
  WaveScratch ws[kTrainWaves];
  double wd[kTrainWaves][4];
};

template <int NT, int EB>
struct Acc {
  v4f c[NT][EB];   // dG_child^T tiles: lane holds n = nt*16 + 4*(lane/16) + i, k = kb*16 + lane%16
  v4f p[NT][EB];   // dG_parent^T tiles
};

// plain (cached) loads: the contraction re-reads the same rows right after
__device__ __forceinline__ float4 ld4(const float *p) {
  return *reinterpret_cast<const float4 *>(p);
}

// The rank-1 updates e_p dA^T of up to four groups' parents as one
// contraction step: row q of the step is pending group q (held in LDS).
template <int NT, int EB>
__device__ __forceinline__ void flush_parents(const TrainArgs &a, WaveScratch &ws,
                                              Acc<NT, EB> &acc, int &np) {
  if (np == 0) return;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
  constexpr int E = EB * 16;
  const bool live = q < np;
  const int32_t tk = ws.ptok[q];
  float av[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) av[nt] = live ? ws.pend[q][nt * 16 + c16] : 0.0f;
  const float *er = a.emb + static_cast<int64_t>(live ? tk : 0) * E + c16;
#pragma unroll
  for (int kb = 0; kb < EB; ++kb) {
    const float b = live ? er[kb * 16] : 0.0f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc.p[nt][kb] = mfma(av[nt], b, acc.p[nt][kb]);
  }
  np = 0;
}

// wave-wide (64-lane) reductions
__device__ __forceinline__ float wave_sum(float v) {
  v = sum16(v);
  return sum_rows(v);
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, xorf(v, 1));
  v = fmaxf(v, xorf(v, 2));
  v = fmaxf(v, xorf(v, 4));
  v = fmaxf(v, xorf(v, 8));
  return max_rows(v);
}

// E-vector x (in LDS) times a staged projection [E][SG]: lane (q, c16) sums
// k in [q E/4, (q+1) E/4) for column nt*16 + c16, then the 4 quarters add up.
template <int NT, int EB>
__device__ __forceinline__ void matvec(const float *x, const float *gs, float (&out)[NT]) {
  constexpr int E = EB * 16, SG = NT * 16 + 4;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
  float4 ev[EB];
#pragma unroll
  for (int t = 0; t < EB; ++t) ev[t] = *reinterpret_cast<const float4 *>(x + q * (E / 4) + 4 * t);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float acc0 = 0.0f;
    const float *gcol = gs + q * (E / 4) * SG + nt * 16 + c16;
#pragma unroll
    for (int t = 0; t < EB; ++t) {
      acc0 = fmaf(ev[t].x, gcol[(4 * t + 0) * SG], acc0);
      acc0 = fmaf(ev[t].y, gcol[(4 * t + 1) * SG], acc0);
      acc0 = fmaf(ev[t].z, gcol[(4 * t + 2) * SG], acc0);
      acc0 = fmaf(ev[t].w, gcol[(4 * t + 3) * SG], acc0);
      __builtin_amdgcn_sched_barrier(0);
    }
    out[nt] = sum_rows(acc0);
  }
}

template <int NT, int EB>
__device__ __forceinline__ void do_group(const TrainArgs &a, TrainLds &s, int wave, int g, float sk,
                                         float inv_sqrt_m, Acc<NT, EB> &acc, int &np,
                                         double (&tot)[4]) {
  constexpr int E = EB * 16, M16 = NT * 16, SG = M16 + 4;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
  const int K = a.K;
  const int p = a.parent[g], d = a.depth[g];
  const int64_t gk = static_cast<int64_t>(g) * K;
  // lane r < K owns child row r for the softmaxes
  const bool own = lane < K;
  const int ctok = own ? a.child[gk + lane] : 0;
  const bool bad = p < 0 || p >= a.V || d < 1 || d > a.L || (own && (ctok < 0 || ctok >= a.V));
  if (__any(bad)) {
    if (lane == 0) atomicOr(a.error_flag, 1u);
    return;
  }
  WaveScratch &ws = s.ws[wave];
  const float *us = s.us + (d - 1) * M16;
  ws.tok[lane] = ctok;

  // parent tower on the VALU
  float abar[NT];
  matvec<NT, EB>(a.emb + static_cast<int64_t>(p) * E, s.gs[0], abar);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) abar[nt] += us[nt * 16 + c16];
  wave_lds_sync();

  // child tower on MFMA, tiles of 16 rows; f and a.b / sqrt(m) go to LDS
#pragma unroll 1
  for (int r0 = 0; r0 < K; r0 += 16) {
    const int row = r0 + c16;
    const bool valid = row < K;
    const float *er = a.emb + static_cast<int64_t>(valid ? ws.tok[row] : 0) * E + 4 * q;
    float4 ev[EB];
#pragma unroll
    for (int kb = 0; kb < EB; ++kb)
      ev[kb] = valid ? ld4(er + kb * 16) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    v4f bb[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) bb[nt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) {
      const float *gb = s.gs[1] + (kb * 16 + 4 * q) * SG + c16;
      const float e4[4] = {ev[kb].x, ev[kb].y, ev[kb].z, ev[kb].w};
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) bb[nt] = mfma(e4[j], gb[j * SG + nt * 16], bb[nt]);
      // keep the next block's LDS operands from being hoisted (register budget)
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float part = 0.0f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) part = fmaf(abar[nt], bb[nt][i] + us[nt * 16 + c16], part);
      const float sum = sum16(part);
      const int r = r0 + 4 * q + i;
      if (c16 == 0 && r < K) {
        ws.f[r] = sk * sum;
        ws.dot[r] = sum * inv_sqrt_m;
      }
    }
  }
  wave_lds_sync();

  // softmaxes over the K children, one row per lane
  const float f = own ? ws.f[lane] : 0.0f;
  const float x = own ? a.logq[gk + lane] + f : -INFINITY;
  const float zt = own ? a.z[gk + lane] : -INFINITY;
  const float y = own && ctok == a.target[g] ? 1.0f : 0.0f;
  const float lse_x = [&] {
    const float mx = wave_max(x);
    return mx + logf(wave_sum(expf(x - mx)));
  }();
  const float lse_z = [&] {
    const float mz = wave_max(zt);
    return mz + logf(wave_sum(expf(zt - mz)));
  }();
  float delta = 0.0f, kl = 0.0f, bce = 0.0f;
  if (own) {
    const float lpt = zt - lse_z, lpth = x - lse_x;
    const float pt = expf(lpt), pth = expf(lpth);
    const float dbce = -a.w1 * y * sigmoid(-f) + (1.0f - y) * sigmoid(f);
    delta = a.c_kl * (pth - pt) + a.c_bce * dbce;
    kl = pt * (lpt - lpth);
    bce = a.w1 * y * softplus(-f) + (1.0f - y) * softplus(f);
  }
  ws.delta[lane] = delta;
  const float sd = wave_sum(delta);
  tot[0] += static_cast<double>(wave_sum(own ? delta * ws.dot[lane] : 0.0f));
  tot[1] += static_cast<double>(wave_sum(kl));
  tot[3] += static_cast<double>(wave_sum(bce));
  wave_lds_sync();

  // dG_child^T += dB^T E_child, four rows per contraction step; the same rows
  // also give sum_r delta_r e_r for the parent-side gradient
  const float *eb = a.emb + c16;
  float wsum[EB];
#pragma unroll
  for (int kb = 0; kb < EB; ++kb) wsum[kb] = 0.0f;
#pragma unroll 2
  for (int r0 = 0; r0 < K; r0 += 4) {
    const int r = r0 + q;
    const bool valid = r < K;
    const float dr = valid ? ws.delta[r] : 0.0f;
    const float *er = eb + static_cast<int64_t>(valid ? ws.tok[r] : 0) * E;
    float av[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) av[nt] = sk * dr * abar[nt];
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) {
      const float b = valid ? er[kb * 16] : 0.0f;
      wsum[kb] = fmaf(dr, b, wsum[kb]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc.c[nt][kb] = mfma(av[nt], b, acc.c[nt][kb]);
    }
  }
  // dL/d(parent tower) = sk (g_child^T sum_r delta_r e_r + u sum_r delta_r)
#pragma unroll
  for (int kb = 0; kb < EB; ++kb) {
    const float v = sum_rows(wsum[kb]);
    if (q == 0) ws.xv[kb * 16 + c16] = v;
  }
  wave_lds_sync();
  float dA[NT];
  matvec<NT, EB>(ws.xv, s.gs[1], dA);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float un = us[nt * 16 + c16];
    dA[nt] = sk * (dA[nt] + un * sd);
    if (q == 0) {
      s.du[wave][(d - 1) * M16 + nt * 16 + c16] += dA[nt] + sk * abar[nt] * sd;
      ws.pend[np][nt * 16 + c16] = dA[nt];   // the parent's rank-1 update waits
    }
  }
  if (lane == 0) ws.ptok[np] = p;
  wave_lds_sync();
  if (++np == 4) flush_parents<NT, EB>(a, ws, acc, np);
}

template <int NT, int EB>
__device__ __forceinline__ void do_pairs(const TrainArgs &a, TrainLds &s, int wave, int tile, float sk,
                         float inv_sqrt_m, Acc<NT, EB> &acc, double (&tot)[4]) {
  constexpr int E = EB * 16, M16 = NT * 16, SG = M16 + 4;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
  WaveScratch &ws = s.ws[wave];
  // forward rows: edge r = c16 is pair tile*8 + r/2, v+ for even r, v- for odd
  const int pr = tile * 8 + (c16 >> 1);
  const int32_t *pe = a.pairs + static_cast<int64_t>(pr < a.P ? pr : 0) * 6 + 3 * (c16 & 1);
  const bool exists = pr < a.P;
  const int ptk = exists ? pe[0] : 0, ctk = exists ? pe[1] : 0, dd = exists ? pe[2] : 1;
  const bool bad_row = exists && (ptk < 0 || ptk >= a.V || ctk < 0 || ctk >= a.V || dd < 1 || dd > a.L);
  if (__any(bad_row)) {
    if (lane == 0) atomicOr(a.error_flag, 1u);
    return;
  }
  if (q == 0) {
    ws.tok[c16] = ptk;
    ws.tok2[c16] = ctk;
    ws.dep[c16] = dd;
  }
  // both towers on MFMA: 16 parent rows through g_parent, 16 child rows through g_child
  v4f pa[NT], pb[NT];
#pragma unroll
  for (int side = 0; side < 2; ++side) {
    const float *er = a.emb + static_cast<int64_t>(side == 0 ? ptk : ctk) * E + 4 * q;
    float4 ev[EB];
#pragma unroll
    for (int kb = 0; kb < EB; ++kb)
      ev[kb] = exists ? ld4(er + kb * 16) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    v4f t[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) t[nt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) {
      const float e4[4] = {ev[kb].x, ev[kb].y, ev[kb].z, ev[kb].w};
      const float *gb = s.gs[side] + (kb * 16 + 4 * q) * SG + c16;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) t[nt] = mfma(e4[j], gb[j * SG + nt * 16], t[nt]);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (side == 0)
        pa[nt] = t[nt];
      else
        pb[nt] = t[nt];
    }
  }
  wave_lds_sync();
  // rows 4q + i of the output: pair tile*8 + 2q + i/2
  float f[4], dot[4], delta[4];
  int drow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    drow[i] = ws.dep[4 * q + i];
    const float *u = s.us + (drow[i] - 1) * M16 + c16;
    float part = 0.0f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      pa[nt][i] += u[nt * 16];
      pb[nt][i] += u[nt * 16];
      part = fmaf(pa[nt][i], pb[nt][i], part);
    }
    const float sum = sum16(part);
    dot[i] = sum * inv_sqrt_m;
    f[i] = sk * sum;
  }
  float loss = 0.0f, dsum = 0.0f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const bool live = tile * 8 + 2 * q + h < a.P;
    const float xm = a.gamma - f[2 * h] + f[2 * h + 1];
    const float t = live ? a.c_pair * sigmoid(xm) : 0.0f;
    loss += live ? softplus(xm) : 0.0f;
    delta[2 * h] = -t;
    delta[2 * h + 1] = t;
    dsum += -t * dot[2 * h] + t * dot[2 * h + 1];
  }
  // every lane of a row holds its row's values; summing the 4 rows gives the tile
  tot[0] += static_cast<double>(sum_rows(dsum));
  tot[2] += static_cast<double>(sum_rows(loss));

  // dY of both towers, depth-embedding gradient (LDS adds: rows of one
  // instruction may share a depth)
  float dA[NT][4], dB[NT][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      dA[nt][i] = sk * delta[i] * pb[nt][i];
      dB[nt][i] = sk * delta[i] * pa[nt][i];
      atomicAdd(&s.du[wave][(drow[i] - 1) * M16 + nt * 16 + c16], dA[nt][i] + dB[nt][i]);
    }
  // parent rows: dG_parent^T += dA^T E_parent, then the child rows
#pragma unroll
  for (int side = 0; side < 2; ++side) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        ws.tile[(4 * q + i) * SG + nt * 16 + c16] = side == 0 ? dA[nt][i] : dB[nt][i];
    wave_lds_sync();
#pragma unroll
    for (int r0 = 0; r0 < 16; r0 += 4) {
      const int r = r0 + q;
      const int tk = side == 0 ? ws.tok[r] : ws.tok2[r];
      const float *er = a.emb + static_cast<int64_t>(tk) * E + c16;
      const bool live = tile * 8 + (r >> 1) < a.P;
      float av[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) av[nt] = live ? ws.tile[r * SG + nt * 16 + c16] : 0.0f;
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) {
        const float b = live ? er[kb * 16] : 0.0f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          if (side == 0)
            acc.p[nt][kb] = mfma(av[nt], b, acc.p[nt][kb]);
          else
            acc.c[nt][kb] = mfma(av[nt], b, acc.c[nt][kb]);
        }
      }
    }
    wave_lds_sync();
  }
}

template <int NT, int EB>
__global__ void __launch_bounds__(kTrainThreads)
train_kernel(TrainArgs a) {
  constexpr int E = EB * 16, M16 = NT * 16, SG = M16 + 4;
  __shared__ TrainLds s;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int q = lane >> 4, c16 = lane & 15;
  const int m = a.m, L = a.L;
  // stage g_parent, g_child (zero columns past m) and u
  for (int i = tid; i < E * SG; i += kTrainThreads) {
    const int k = i / SG, n = i % SG;
    const bool in = n < m;
    s.gs[0][i] = in ? a.theta[k * m + n] : 0.0f;
    s.gs[1][i] = in ? a.theta[E * m + k * m + n] : 0.0f;
  }
  for (int i = tid; i < L * M16; i += kTrainThreads) {
    const int l = i / M16, n = i % M16;
    s.us[i] = n < m ? a.theta[2 * E * m + l * m + n] : 0.0f;
  }
  for (int i = tid; i < kTrainWaves * kMaxLM; i += kTrainThreads) (&s.du[0][0])[i] = 0.0f;
  const float inv_sqrt_m = 1.0f / sqrtf(static_cast<float>(m));
  const float sk = a.theta[2 * E * m + L * m] * inv_sqrt_m;
  __syncthreads();

  Acc<NT, EB> acc;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int kb = 0; kb < EB; ++kb) acc.c[nt][kb] = acc.p[nt][kb] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  int np = 0;
  double tot[4] = {0.0, 0.0, 0.0, 0.0};

  // cost-weighted contiguous share: groups cost 1, pair tiles 2
  const int64_t T = (a.P + 7) / 8;
  const int64_t C = static_cast<int64_t>(a.G) + 2 * T;
  const int64_t W = static_cast<int64_t>(gridDim.x) * kTrainWaves;
  const int64_t w = static_cast<int64_t>(blockIdx.x) * kTrainWaves + wave;
  const int64_t lo = w * C / W, hi = (w + 1) * C / W;
  for (int64_t g = lo; g < hi && g < a.G; ++g)
    do_group<NT, EB>(a, s, wave, static_cast<int>(g), sk, inv_sqrt_m, acc, np, tot);
  flush_parents<NT, EB>(a, s.ws[wave], acc, np);
  const int64_t t0 = lo > a.G ? (lo - a.G + 1) / 2 : 0;
  const int64_t t1 = hi > a.G ? (hi - a.G + 1) / 2 : 0;
  for (int64_t t = t0; t < t1 && t < T; ++t)
    do_pairs<NT, EB>(a, s, wave, static_cast<int>(t), sk, inv_sqrt_m, acc, tot);

  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) s.wd[wave][j] = tot[j];
  }
  __syncthreads();
  // block sum of the waves' accumulators, in wave order: [child | parent] x [n][k]
  float *red = &s.gs[0][0];
  for (int wv = 0; wv < kTrainWaves; ++wv) {
    if (wave == wv) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int kb = 0; kb < EB; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int idx = (nt * 16 + 4 * q + i) * E + kb * 16 + c16;
            red[idx] = (wv ? red[idx] : 0.0f) + acc.c[nt][kb][i];
            red[M16 * E + idx] = (wv ? red[M16 * E + idx] : 0.0f) + acc.p[nt][kb][i];
          }
    }
    __syncthreads();
  }
  const int n_g = 2 * E * m + L * m;
  float *out = a.part_g + static_cast<int64_t>(blockIdx.x) * n_g;
  for (int i = tid; i < n_g; i += kTrainThreads) {
    float v;
    if (i < 2 * E * m) {
      const int kind = i / (E * m), r = i % (E * m), k = r / m, n = r % m;
      v = red[(kind == 0 ? M16 * E : 0) + n * E + k];
    } else {
      const int r = i - 2 * E * m, l = r / m, n = r % m;
      v = 0.0f;
      for (int wv = 0; wv < kTrainWaves; ++wv) v += s.du[wv][l * M16 + n];
    }
    out[i] = v;
  }
  if (tid < 4) {
    double v = 0.0;
    for (int wv = 0; wv < kTrainWaves; ++wv) v += s.wd[wv][tid];
    a.part_d[static_cast<int64_t>(blockIdx.x) * 4 + tid] = v;
  }
}

struct UpdateArgs {
  float *theta, *m1, *m2, *grad_out;
  const float *part_g;
  const double *part_d;
  double *loss;
  int n_params, n_g, blocks, G, P, K;
  double lr, wd, beta1, beta2, eps, bc1, bc2;
  double lambda_kl, lambda_pair, lambda_bce;
};

__global__ void __launch_bounds__(256) update_kernel(UpdateArgs u) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i == 0 && u.loss) {
    double kl = 0.0, pr = 0.0, bce = 0.0;
    for (int b = 0; b < u.blocks; ++b) {
      kl += u.part_d[b * 4 + 1];
      pr += u.part_d[b * 4 + 2];
      bce += u.part_d[b * 4 + 3];
    }
    kl = u.G ? kl / u.G : 0.0;
    pr = u.P ? pr / u.P : 0.0;
    bce = u.G ? bce / (static_cast<double>(u.G) * u.K) : 0.0;
    u.loss[0] = u.lambda_kl * kl + u.lambda_pair * pr + u.lambda_bce * bce;
    u.loss[1] = kl;
    u.loss[2] = pr;
    u.loss[3] = bce;
  }
  if (i >= u.n_params) return;
  double g = 0.0;
  if (i < u.n_g) {
    for (int b = 0; b < u.blocks; ++b) g += static_cast<double>(u.part_g[static_cast<int64_t>(b) * u.n_g + i]);
  } else {
    for (int b = 0; b < u.blocks; ++b) g += u.part_d[b * 4];
  }
  if (u.grad_out) u.grad_out[i] = static_cast<float>(g);
  double th = static_cast<double>(u.theta[i]) * (1.0 - u.lr * u.wd);
  const double m1 = u.beta1 * static_cast<double>(u.m1[i]) + (1.0 - u.beta1) * g;
  const double m2 = u.beta2 * static_cast<double>(u.m2[i]) + (1.0 - u.beta2) * g * g;
  th -= u.lr * (m1 / u.bc1) / (sqrt(m2 / u.bc2) + u.eps);
  u.theta[i] = static_cast<float>(th);
  u.m1[i] = static_cast<float>(m1);
  u.m2[i] = static_cast<float>(m2);
}

template <int NT, int EB>
bool launch_train_t(const TrainArgs &a, int nt, int eb, int blocks, hipStream_t stream) {
  if (nt != NT || eb != EB) return false;
  hipLaunchKernelGGL((train_kernel<NT, EB>), dim3(blocks), dim3(kTrainThreads), 0, stream, a);
  return true;
}

// the instantiated shapes: E in {32, 64, 128} with E * ceil(m/16) * 16 <= 4096
bool dispatch_train(const TrainArgs &a, int nt, int eb, int blocks, hipStream_t stream) {
  return launch_train_t<1, 2>(a, nt, eb, blocks, stream) ||
         launch_train_t<1, 4>(a, nt, eb, blocks, stream) ||
         launch_train_t<1, 8>(a, nt, eb, blocks, stream) ||
         launch_train_t<2, 2>(a, nt, eb, blocks, stream) ||
         launch_train_t<2, 4>(a, nt, eb, blocks, stream) ||
         launch_train_t<2, 8>(a, nt, eb, blocks, stream) ||
         launch_train_t<3, 2>(a, nt, eb, blocks, stream) ||
         launch_train_t<3, 4>(a, nt, eb, blocks, stream) ||
         launch_train_t<4, 2>(a, nt, eb, blocks, stream) ||
         launch_train_t<4, 4>(a, nt, eb, blocks, stream);
}

}  // namespace

int tdes_blocks(int G, int P) {
  const int64_t cost = static_cast<int64_t>(G) + 2 * ((static_cast<int64_t>(P) + 7) / 8);
  int64_t b = (cost + 2 * kTrainWaves - 1) / (2 * kTrainWaves);   // >= 2 items per wave
  if (b < 1) b = 1;
  if (b > kTdesMaxBlocks) b = kTdesMaxBlocks;
  return static_cast<int>(b);
}

bool tdes_shape_supported(int E, int m, int L, int K) {
  const int m16 = (m + 15) / 16 * 16;
  const bool e_ok = E == 32 || E == 64 || E == 128;
  return e_ok && m >= 1 && m <= kMaxScoreDim && E * m16 <= kMaxEM && L >= 1 && L * m16 <= kMaxLM &&
         K >= 1 && K <= kMaxK && E * (m16 + 4) <= kMaxGs;
}

hipError_t launch_tdes_step(graft_tdes *t, const float *emb, const graft_tdes_batch *b,
                            const graft_tdes_hyper *h, int32_t step, float *theta, float *m1,
                            float *m2, double *loss, float *grad, hipStream_t stream) {
  const graft_tdes_dims &d = t->dims;
  const int E = d.emb_dim, m = d.score_dim, L = d.num_pos, K = d.top_k;
  const int G = b->n_groups, P = b->n_pairs;
  const int blocks = tdes_blocks(G, P);
  TrainArgs a;
  a.emb = emb;
  a.theta = theta;
  a.V = d.vocab;
  a.E = E;
  a.m = m;
  a.L = L;
  a.K = K;
  a.G = G;
  a.P = P;
  a.parent = b->parent;
  a.depth = b->depth;
  a.child = b->child;
  a.target = b->target;
  a.pairs = b->pairs;
  a.logq = b->logq;
  a.z = b->z_target;
  a.c_kl = G ? static_cast<float>(static_cast<double>(h->lambda_kl) / G) : 0.0f;
  a.c_bce = G ? static_cast<float>(static_cast<double>(h->lambda_bce) / (static_cast<double>(G) * K)) : 0.0f;
  a.c_pair = P ? static_cast<float>(static_cast<double>(h->lambda_pair) / P) : 0.0f;
  a.gamma = h->gamma;
  a.w1 = h->w1;
  a.part_g = t->part_g;
  a.part_d = t->part_d;
  a.error_flag = t->error_flag;
  if (!dispatch_train(a, (m + 15) / 16, E / 16, blocks, stream)) return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  UpdateArgs u;
  u.theta = theta;
  u.m1 = m1;
  u.m2 = m2;
  u.grad_out = grad;
  u.part_g = t->part_g;
  u.part_d = t->part_d;
  u.loss = loss;
  u.n_params = 2 * E * m + L * m + 1;
  u.n_g = 2 * E * m + L * m;
  u.blocks = blocks;
  u.G = G;
  u.P = P;
  u.K = K;
  u.lr = h->lr;
  u.wd = h->weight_decay;
  u.beta1 = h->beta1;
  u.beta2 = h->beta2;
  u.eps = h->eps;
  u.bc1 = 1.0 - std::pow(static_cast<double>(h->beta1), step);
  u.bc2 = 1.0 - std::pow(static_cast<double>(h->beta2), step);
  u.lambda_kl = h->lambda_kl;
  u.lambda_pair = h->lambda_pair;
  u.lambda_bce = h->lambda_bce;
  hipLaunchKernelGGL(update_kernel, dim3((u.n_params + 255) / 256), dim3(256), 0, stream, u);
  return hipGetLastError();
}

}  // namespace graft
