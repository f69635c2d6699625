// k_tdes_train.hip -- one training step of the TDES edge scorer (the paper's
// Target-Distilled Edge Scoring section: scorer eq. tdes-bitower; objectives
// KL, pairwise margin and class-balanced BCE, summed by eq. tdes-training;
// AdamW as in the training setup of the experiments).
//
// Rows.  Every edge of the batch contributes a parent-tower row and a
// child-tower row: the K children and the parent of each group (the parent
// row is shared by its K edges), and both edges of each pair.  With the
// towers a = g_p(e_p) + u_d, b = g_c(e_c) + u_d and f = s a.b / sqrt(m), the
// weight gradients are contractions over rows,
//   dL/dg_parent = sum over parent rows of e (dL/da)^T,
//   dL/dg_child  = sum over child rows of e (dL/db)^T.
//
// loss_kernel (one wave per group or tile of 8 pairs): gathers the item's
//   embedding rows (16-byte loads), projects them on MFMA
//   (v_mfma_f32_16x16x4_f32, 16 rows x 16 score dimensions per instruction;
//   g_parent and g_child staged in LDS), forms f, the objectives and dL/df,
//   and writes dL/da, dL/db of every row (fp32, m padded to a multiple of 16)
//   plus per-block sums of the depth-embedding and scale gradients and of the
//   objectives.  Few registers per wave: many waves in flight hide the gathers.
// wgrad_kernel: the two contractions on MFMA, 4 rows per instruction, over
//   contiguous row chunks (the embedding rows come back from L2 / MALL, 16
//   bytes per lane); per-block partial gradients.
// update_kernel: sums every partial in fp64 in a fixed order (a step is
//   deterministic), then applies AdamW to every parameter.
#include <cmath>

#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kLossWaves = 4;
constexpr int kLossThreads = kLossWaves * kWave;
constexpr int kGradWaves = 8;
constexpr int kGradThreads = kGradWaves * kWave;
constexpr int kGradRowsPerWave = 32;
constexpr int kGradRows = kGradWaves * kGradRowsPerWave;   // rows per wgrad block
constexpr int kMaxEM = 4096;          // E * M16, M16 = m rounded up to 16
constexpr int kMaxLM = 1024;          // L * M16

typedef float v4f __attribute__((ext_vector_type(4)));

struct TrainArgs {
  const float *emb;      // [V, E]
  const float *theta;    // [gp E*m | gc E*m | u L*m | s]
  int V, E, m, L, K;
  int G, P;
  const int32_t *parent, *depth, *child, *target, *pairs;
  const float *logq, *z;
  float c_kl, c_bce, c_pair, gamma, w1;
  float *dyc;            // [G*K + 2P, M16] dL/db of the child-tower rows
  float *dyp;            // [G + 2P, M16] dL/da of the parent-tower rows
  float *part_u;         // L*m per loss block (chunked)
  double *part_d;        // [loss blocks, 4]: ds, sum KL, sum pair, sum BCE
  float *part_w;         // E*m per child-side then parent-side wgrad block (chunked)
  uint32_t *error_flag;
};

__device__ __forceinline__ float xorf(float v, int m) {
  return __uint_as_float(xor_lane(__float_as_uint(v), m));
}
// sum over the 16 lanes of a row of lanes (equal lane / 16)
__device__ __forceinline__ float sum16(float v) {
  v += xorf(v, 1);
  v += xorf(v, 2);
  v += xorf(v, 4);
  v += xorf(v, 8);
  return v;
}
// sum / max over the 4 rows of lanes (equal lane % 16)
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
__device__ __forceinline__ float wave_sum(float v) { return sum_rows(sum16(v)); }
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, xorf(v, 1));
  v = fmaxf(v, xorf(v, 2));
  v = fmaxf(v, xorf(v, 4));
  v = fmaxf(v, xorf(v, 8));
  return max_rows(v);
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
__device__ __forceinline__ float4 ld4(const float *p) {
  return *reinterpret_cast<const float4 *>(p);
}

// Block partials are stored chunked, [n / kChunk][blocks][kChunk]: a block
// writes kChunk consecutive values per chunk and the update reads each chunk
// of all blocks as one contiguous run.
constexpr int kChunk = 32;
__host__ __device__ __forceinline__ int64_t chunked(int i, int blocks, int b) {
  return (static_cast<int64_t>(i / kChunk) * blocks + b) * kChunk + i % kChunk;
}
__host__ __device__ __forceinline__ int64_t chunked_size(int n, int blocks) {
  return static_cast<int64_t>((n + kChunk - 1) / kChunk) * blocks * kChunk;
}

// 16 rows of E fp32 embedding entries times a staged projection [E][SG]: lane
// (q, c16) supplies entries kb*16 + 4q + j of its row (row c16 of the tile);
// the result holds rows 4q + i, column nt*16 + c16 in component i.
template <int EB>
__device__ __forceinline__ void load16(const float *row, bool valid, float4 (&ev)[EB]) {
  const int q = lane_id() >> 4;
#pragma unroll
  for (int kb = 0; kb < EB; ++kb)
    ev[kb] = valid ? ld4(row + kb * 16 + 4 * q) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
}
template <int NT, int EB>
__device__ __forceinline__ void mma16(const float4 (&ev)[EB], const float *gs, v4f (&y)[NT]) {
  constexpr int SG = NT * 16 + 4;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) y[nt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int kb = 0; kb < EB; ++kb) {
    const float *gb = gs + (kb * 16 + 4 * q) * SG + c16;
    const float e4[4] = {ev[kb].x, ev[kb].y, ev[kb].z, ev[kb].w};
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) y[nt] = mfma(e4[j], gb[j * SG + nt * 16], y[nt]);
  }
}
template <int NT, int EB>
__device__ __forceinline__ void project16(const float *row, bool valid, const float *gs, v4f (&y)[NT]) {
  float4 ev[EB];
  load16<EB>(row, valid, ev);
  mma16<NT, EB>(ev, gs, y);
}

// LDS of loss_kernel (dynamic): gs0, gs1 [E][SG] | us [L][M16] |
// du [waves][L][M16] | per wave delta, f, dot [64 each] | wd [waves][4] (double)
struct LossLds {
  float *gs0, *gs1, *us, *du, *wsf;
  double *wd;
};

__device__ __forceinline__ LossLds loss_lds(char *base, int E, int M16, int L) {
  LossLds s;
  const int SG = M16 + 4;
  float *p = reinterpret_cast<float *>(base);
  s.gs0 = p;
  s.gs1 = p + E * SG;
  s.us = s.gs1 + E * SG;
  s.du = s.us + L * M16;
  s.wsf = s.du + kLossWaves * L * M16;
  s.wd = reinterpret_cast<double *>(s.wsf + kLossWaves * 3 * kMaxK);
  return s;
}

template <int NT, int EB, int RT>
__device__ __forceinline__ void group_item(const TrainArgs &a, const LossLds &s, int wave, int g,
                                           float sk, float inv_sqrt_m, double (&tot)[4]) {
  constexpr int E = EB * 16, M16 = NT * 16;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
  const int K = a.K;
  const int64_t gk = static_cast<int64_t>(g) * K;
  const int p = a.parent[g], d = a.depth[g];
  // lane r < K owns child row r for the softmaxes; its inputs load early
  const bool own = lane < K;
  const int ctok = own ? a.child[gk + lane] : 0;
  const float lq = own ? a.logq[gk + lane] : 0.0f;
  const float zt = own ? a.z[gk + lane] : -INFINITY;
  const int tgt = a.target[g];
  float *dyc = a.dyc + gk * M16;
  float *dyp = a.dyp + static_cast<int64_t>(g) * M16;
  const bool bad = p < 0 || p >= a.V || d < 1 || d > a.L || (own && (ctok < 0 || ctok >= a.V));
  if (__any(bad)) {
    // dropped: zero rows keep the contractions exact for the rest
    for (int i = lane; i < K * M16; i += kWave) dyc[i] = 0.0f;
    if (lane < M16) dyp[lane] = 0.0f;
    if (lane == 0) atomicOr(a.error_flag, 1u);
    return;
  }
  float *delta = s.wsf + wave * 3 * kMaxK, *fs = delta + kMaxK, *dots = fs + kMaxK;
  const float *us = s.us + (d - 1) * M16;

  // parent tower on the VALU (one row): lane (q, c16) sums entries
  // kb*16 + 4q + j for column nt*16 + c16, then the 4 rows of lanes add up.
  // Its loads go out with those of the first child tile.
  float4 evc0[EB];
  float abar[NT];
  {
    float4 evp[EB];
    load16<EB>(a.emb + static_cast<int64_t>(p) * E, true, evp);
    load16<EB>(a.emb + static_cast<int64_t>(__shfl(ctok, c16)) * E, c16 < K, evc0);
    constexpr int SG = M16 + 4;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float acc0 = 0.0f;
#pragma unroll
      for (int kb = 0; kb < EB; ++kb) {
        const float *gcol = s.gs0 + (kb * 16 + 4 * q) * SG + nt * 16 + c16;
        acc0 = fmaf(evp[kb].x, gcol[0], acc0);
        acc0 = fmaf(evp[kb].y, gcol[SG], acc0);
        acc0 = fmaf(evp[kb].z, gcol[2 * SG], acc0);
        acc0 = fmaf(evp[kb].w, gcol[3 * SG], acc0);
      }
      abar[nt] = sum_rows(acc0) + us[nt * 16 + c16];
    }
  }

  // child tower, RT tiles of 16 rows (kept for dL/da)
  v4f bb[RT][NT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) bb[rt][nt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    if (rt * 16 < K) {
      const int row = rt * 16 + c16;
      if (rt == 0) {
        mma16<NT, EB>(evc0, s.gs1, bb[0]);
      } else {
        const int tok = __shfl(ctok, row);
        project16<NT, EB>(a.emb + static_cast<int64_t>(tok) * E, row < K, s.gs1, bb[rt]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float part = 0.0f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          bb[rt][nt][i] += us[nt * 16 + c16];
          part = fmaf(abar[nt], bb[rt][nt][i], part);
        }
        const float sum = sum16(part);
        const int r = rt * 16 + 4 * q + i;
        if (c16 == 0 && r < K) {
          fs[r] = sk * sum;
          dots[r] = sum * inv_sqrt_m;
        }
      }
    }
  }
  wave_lds_sync();

  // softmaxes over the K children, one row per lane
  const float f = own ? fs[lane] : 0.0f;
  const float x = own ? lq + f : -INFINITY;
  const float y = own && ctok == tgt ? 1.0f : 0.0f;
  const float mx = wave_max(x), mz = wave_max(zt);
  const float lse_x = mx + logf(wave_sum(own ? expf(x - mx) : 0.0f));
  const float lse_z = mz + logf(wave_sum(own ? expf(zt - mz) : 0.0f));
  float dl = 0.0f, kl = 0.0f, bce = 0.0f;
  if (own) {
    const float lpt = zt - lse_z, lpth = x - lse_x;
    const float pt = expf(lpt), pth = expf(lpth);
    const float dbce = -a.w1 * y * sigmoid(-f) + (1.0f - y) * sigmoid(f);
    dl = a.c_kl * (pth - pt) + a.c_bce * dbce;
    kl = pt * (lpt - lpth);
    bce = a.w1 * y * softplus(-f) + (1.0f - y) * softplus(f);
  }
  delta[lane] = dl;
  const float sd = wave_sum(dl);
  tot[0] += static_cast<double>(wave_sum(own ? dl * dots[lane] : 0.0f));
  tot[1] += static_cast<double>(wave_sum(kl));
  tot[3] += static_cast<double>(wave_sum(bce));
  wave_lds_sync();

  // dL/db_r = sk delta_r abar (lanes of row q of lanes take rows q, q + 4, ...)
  for (int r = q; r < K; r += 4) {
    const float c = sk * delta[r];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) dyc[r * M16 + nt * 16 + c16] = c * abar[nt];
  }
  // dL/da = sk sum_r delta_r bbar_r; the depth embedding gets dL/da + sum_r dL/db_r
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float part = 0.0f;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = rt * 16 + 4 * q + i;
        part = fmaf(r < K ? delta[r] : 0.0f, bb[rt][nt][i], part);
      }
    const float dA = sk * sum_rows(part);
    if (q == 0) {
      dyp[nt * 16 + c16] = dA;
      s.du[(wave * a.L + d - 1) * M16 + nt * 16 + c16] += dA + sk * abar[nt] * sd;
    }
  }
  wave_lds_sync();
}

template <int NT, int EB>
__device__ __forceinline__ void pair_item(const TrainArgs &a, const LossLds &s, int wave, int tile,
                                          float sk, float inv_sqrt_m, double (&tot)[4]) {
  constexpr int E = EB * 16, M16 = NT * 16;
  const int lane = lane_id(), q = lane >> 4, c16 = lane & 15;
  // edge r = c16 of the tile: pair tile*8 + r/2, v+ for even r, v- for odd
  const int pr = tile * 8 + (c16 >> 1);
  const bool exists = pr < a.P;
  const int32_t *pe = a.pairs + static_cast<int64_t>(exists ? pr : 0) * 6 + 3 * (c16 & 1);
  const int ptk = exists ? pe[0] : 0, ctk = exists ? pe[1] : 0, dd = exists ? pe[2] : 1;
  const int64_t pbase = a.G + static_cast<int64_t>(tile) * 16;   // dyp row of edge 0
  const int64_t cbase = static_cast<int64_t>(a.G) * a.K + static_cast<int64_t>(tile) * 16;
  const bool bad_row = exists && (ptk < 0 || ptk >= a.V || ctk < 0 || ctk >= a.V || dd < 1 || dd > a.L);
  if (__any(bad_row)) {
    for (int i = lane; i < 16 * M16; i += kWave) {
      if (tile * 8 + (i / M16) / 2 < a.P) {
        a.dyp[pbase * M16 + i] = 0.0f;
        a.dyc[cbase * M16 + i] = 0.0f;
      }
    }
    if (lane == 0) atomicOr(a.error_flag, 1u);
    return;
  }
  v4f pa[NT], pb[NT];
  {
    float4 evp[EB], evc[EB];
    load16<EB>(a.emb + static_cast<int64_t>(ptk) * E, exists, evp);
    load16<EB>(a.emb + static_cast<int64_t>(ctk) * E, exists, evc);
    mma16<NT, EB>(evp, s.gs0, pa);
    mma16<NT, EB>(evc, s.gs1, pb);
  }
  // output rows 4q + i: pair tile*8 + 2q + i/2
  float f[4], dot[4], dl[4];
  int drow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    drow[i] = __shfl(dd, 4 * q + i);
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
    dl[2 * h] = -t;
    dl[2 * h + 1] = t;
    dsum += -t * dot[2 * h] + t * dot[2 * h + 1];
  }
  // each lane holds its row of lanes' two pairs: the 4 rows of lanes sum to the tile
  tot[0] += static_cast<double>(sum_rows(dsum));
  tot[2] += static_cast<double>(sum_rows(loss));
  // dL/da = sk delta bbar, dL/db = sk delta abar; the depth embedding gets both
  // (LDS adds: rows of one instruction may share a depth)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * q + i;
    const bool live = tile * 8 + r / 2 < a.P;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const float dA = sk * dl[i] * pb[nt][i], dB = sk * dl[i] * pa[nt][i];
      if (live) {
        a.dyp[(pbase + r) * M16 + nt * 16 + c16] = dA;
        a.dyc[(cbase + r) * M16 + nt * 16 + c16] = dB;
        atomicAdd(&s.du[(wave * a.L + drow[i] - 1) * M16 + nt * 16 + c16], dA + dB);
      }
    }
  }
}

template <int NT, int EB, int RT>
__global__ void __launch_bounds__(kLossThreads)
loss_kernel(TrainArgs a) {
  constexpr int E = EB * 16, M16 = NT * 16, SG = M16 + 4;
  extern __shared__ __align__(16) char lds_raw[];
  const LossLds s = loss_lds(lds_raw, E, M16, a.L);
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int m = a.m, L = a.L;
  // stage g_parent, g_child as [E][SG] (columns m.. zero): with m a multiple
  // of 4 every thread's float4 loads go out together
  if (m % 4 == 0) {
    const int n4 = E * m / 4;
    for (int i = tid; i < E * SG; i += kLossThreads) {
      const int n = i % SG;
      if (n >= m) s.gs0[i] = s.gs1[i] = 0.0f;
    }
    constexpr int kPer = (E * M16 / 4 + kLossThreads - 1) / kLossThreads;
    float4 v0[kPer], v1[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int v = tid + j * kLossThreads;
      if (v < n4) {
        v0[j] = ld4(a.theta + 4 * v);
        v1[j] = ld4(a.theta + E * m + 4 * v);
      }
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int v = tid + j * kLossThreads;
      if (v < n4) {
        const int k = 4 * v / m, n = 4 * v % m;
        float *d0 = s.gs0 + k * SG + n, *d1 = s.gs1 + k * SG + n;
        d0[0] = v0[j].x, d0[1] = v0[j].y, d0[2] = v0[j].z, d0[3] = v0[j].w;
        d1[0] = v1[j].x, d1[1] = v1[j].y, d1[2] = v1[j].z, d1[3] = v1[j].w;
      }
    }
  } else {
    for (int i = tid; i < E * SG; i += kLossThreads) {
      const int k = i / SG, n = i % SG;
      const bool in = n < m;
      s.gs0[i] = in ? a.theta[k * m + n] : 0.0f;
      s.gs1[i] = in ? a.theta[E * m + k * m + n] : 0.0f;
    }
  }
  for (int i = tid; i < L * M16; i += kLossThreads) {
    const int l = i / M16, n = i % M16;
    s.us[i] = n < m ? a.theta[2 * E * m + l * m + n] : 0.0f;
  }
  for (int i = tid; i < kLossWaves * L * M16; i += kLossThreads) s.du[i] = 0.0f;
  const float inv_sqrt_m = 1.0f / sqrtf(static_cast<float>(m));
  const float sk = a.theta[2 * E * m + L * m] * inv_sqrt_m;
  __syncthreads();

  double tot[4] = {0.0, 0.0, 0.0, 0.0};
  const int T = (a.P + 7) / 8;
  const int items = a.G + T;
  const int W = gridDim.x * kLossWaves;
  for (int it = blockIdx.x * kLossWaves + wave; it < items; it += W) {
    if (it < a.G)
      group_item<NT, EB, RT>(a, s, wave, it, sk, inv_sqrt_m, tot);
    else
      pair_item<NT, EB>(a, s, wave, it - a.G, sk, inv_sqrt_m, tot);
  }
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) s.wd[wave * 4 + j] = tot[j];
  }
  __syncthreads();
  for (int i = tid; i < L * m; i += kLossThreads) {
    const int l = i / m, n = i % m;
    float v = 0.0f;
    for (int wv = 0; wv < kLossWaves; ++wv) v += s.du[(wv * L + l) * M16 + n];
    a.part_u[chunked(i, gridDim.x, blockIdx.x)] = v;
  }
  if (tid < 4) {
    double v = 0.0;
    for (int wv = 0; wv < kLossWaves; ++wv) v += s.wd[wv * 4 + tid];
    a.part_d[static_cast<int64_t>(blockIdx.x) * 4 + tid] = v;
  }
}

// Token of row `row` of one side: child side = the children of the groups,
// then the child of every pair edge; parent side = the parents of the groups,
// then the parent of every pair edge (edge 2i is v+ of pair i, 2i + 1 its v-).
__device__ __forceinline__ int row_token(const TrainArgs &a, int side, int64_t row) {
  const int64_t first = side == 0 ? static_cast<int64_t>(a.G) * a.K : a.G;
  if (row < first) return side == 0 ? a.child[row] : a.parent[row];
  const int64_t e = row - first;
  return a.pairs[(e >> 1) * 6 + 3 * (e & 1) + (side == 0 ? 1 : 0)];
}

// dL/dg = sum over the rows of one side of e_row (dL/dy_row)^T, 4 rows per
// instruction.  Lane (q, c16) loads 16 bytes of embedding row 4s + q,
// entries 64h + 4 c16 + j, so tile (nt, 4h + j) of the transposed gradient
// holds n = nt*16 + 4q + i (component i), k = 64h + 4 c16 + j.
template <int NT, int EB>
__global__ void __launch_bounds__(kGradThreads)
wgrad_kernel(TrainArgs a, int child_blocks) {
  constexpr int E = EB * 16, M16 = NT * 16, KH = (E + 63) / 64;
  __shared__ float red[kMaxEM];
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int q = lane >> 4, c16 = lane & 15;
  const int side = blockIdx.x < child_blocks ? 0 : 1;
  const int blk = side == 0 ? blockIdx.x : blockIdx.x - child_blocks;
  const int64_t rows = side == 0 ? static_cast<int64_t>(a.G) * a.K + 2 * static_cast<int64_t>(a.P)
                                 : static_cast<int64_t>(a.G) + 2 * static_cast<int64_t>(a.P);
  const float *dy = side == 0 ? a.dyc : a.dyp;
  v4f acc[NT][4 * KH];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int t = 0; t < 4 * KH; ++t) acc[nt][t] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  const int64_t r0 = static_cast<int64_t>(blk) * kGradRows + wave * kGradRowsPerWave;
  // the tokens of the wave's rows, one per lane, in one round trip
  int mytok = -1;
  if (lane < kGradRowsPerWave && r0 + lane < rows) mytok = row_token(a, side, r0 + lane);
  const bool kin = 4 * c16 < E;   // E = 32 uses half the lanes of a 64-entry block
#pragma unroll 4
  for (int st = 0; st < kGradRowsPerWave; st += 4) {
    const int64_t r = r0 + st + q;
    const int tok = __shfl(mytok, st + q);
    const bool live = r < rows && tok >= 0 && tok < a.V;
    const float *er = a.emb + static_cast<int64_t>(live ? tok : 0) * E + 4 * c16;
    const float *yr = dy + (live ? r : 0) * M16 + c16;
    float av[NT];
    float4 ev[KH];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) av[nt] = live ? yr[nt * 16] : 0.0f;
#pragma unroll
    for (int h = 0; h < KH; ++h)
      ev[h] = live && kin ? ld4(er + 64 * h) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int h = 0; h < KH; ++h) {
        acc[nt][4 * h + 0] = mfma(av[nt], ev[h].x, acc[nt][4 * h + 0]);
        acc[nt][4 * h + 1] = mfma(av[nt], ev[h].y, acc[nt][4 * h + 1]);
        acc[nt][4 * h + 2] = mfma(av[nt], ev[h].z, acc[nt][4 * h + 2]);
        acc[nt][4 * h + 3] = mfma(av[nt], ev[h].w, acc[nt][4 * h + 3]);
      }
  }
  // block sum in wave order into red[n][k] (one wave at a time measured faster
  // than four LDS slots added pairwise)
  for (int wv = 0; wv < kGradWaves; ++wv) {
    if (wave == wv && kin) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int t = 0; t < 4 * KH; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int k = 64 * (t / 4) + 4 * c16 + (t % 4);
            const int idx = (nt * 16 + 4 * q + i) * E + k;
            if (k < E) red[idx] = (wv ? red[idx] : 0.0f) + acc[nt][t][i];
          }
    }
    __syncthreads();
  }
  const int m = a.m, em = E * m;
  const int nb = side == 0 ? child_blocks : gridDim.x - child_blocks;
  float *out = a.part_w + (side == 0 ? 0 : chunked_size(em, child_blocks));
  for (int i = tid; i < em; i += kGradThreads) {
    const int idx = (i % m) * E + i / m;
    const float v = red[idx];
    out[chunked(i, nb, blk)] = v;
  }
}

struct UpdateArgs {
  float *theta, *m1, *m2, *grad_out;
  const float *part_u, *part_w;
  const double *part_d;
  double *loss;
  int E, m, L, n_params, loss_blocks, child_blocks, parent_blocks, G, P, K;
  double lr, wd, beta1, beta2, eps, bc1, bc2;
  double lambda_kl, lambda_pair, lambda_bce;
};

// Block r < 2 cw + cu (cw, cu: chunks of E*m and L*m) updates the kChunk
// parameters of one chunk of g_parent, g_child or u: thread (slice, o) sums
// blocks slice, slice + kUpdSlices, ... of parameter o, then the slices add
// in order.  The last block does the scale and the objectives with fixed-order
// tree sums.  Every sum is fp64 and deterministic.
constexpr int kUpdSlices = 32;
constexpr int kUpdThreads = kChunk * kUpdSlices;

__device__ __forceinline__ void adamw(const UpdateArgs &u, int i, double g) {
  if (u.grad_out) u.grad_out[i] = static_cast<float>(g);
  double th = static_cast<double>(u.theta[i]) * (1.0 - u.lr * u.wd);
  const double m1 = u.beta1 * static_cast<double>(u.m1[i]) + (1.0 - u.beta1) * g;
  const double m2 = u.beta2 * static_cast<double>(u.m2[i]) + (1.0 - u.beta2) * g * g;
  th -= u.lr * (m1 / u.bc1) / (sqrt(m2 / u.bc2) + u.eps);
  u.theta[i] = static_cast<float>(th);
  u.m1[i] = static_cast<float>(m1);
  u.m2[i] = static_cast<float>(m2);
}

__global__ void __launch_bounds__(kUpdThreads) update_kernel(UpdateArgs u) {
  __shared__ double red[kUpdSlices][kChunk];
  __shared__ double tree[4][kTdesMaxLossBlocks];
  const int tid = threadIdx.x;
  const int em = u.E * u.m, lm = u.L * u.m;
  const int cw = (em + kChunk - 1) / kChunk, cu = (lm + kChunk - 1) / kChunk;
  const int r = blockIdx.x;
  if (r < 2 * cw + cu) {
    const int o = tid % kChunk, sl = tid / kChunk;
    const float *src;
    int nb, c, base, n;
    if (r < cw) {            // g_parent: parent-side wgrad blocks
      src = u.part_w + chunked_size(em, u.child_blocks);
      nb = u.parent_blocks, c = r, base = 0, n = em;
    } else if (r < 2 * cw) { // g_child: child-side wgrad blocks
      src = u.part_w;
      nb = u.child_blocks, c = r - cw, base = em, n = em;
    } else {                 // depth embedding: loss blocks
      src = u.part_u;
      nb = u.loss_blocks, c = r - 2 * cw, base = 2 * em, n = lm;
    }
    const float *run = src + static_cast<int64_t>(c) * nb * kChunk + o;
    double g = 0.0;
#pragma unroll 8
    for (int b = sl; b < nb; b += kUpdSlices) g += static_cast<double>(run[static_cast<int64_t>(b) * kChunk]);
    red[sl][o] = g;
    __syncthreads();
    const int i = c * kChunk + o;
    if (sl != 0 || i >= n) return;
    g = 0.0;
    for (int k = 0; k < kUpdSlices; ++k) g += red[k][o];
    adamw(u, base + i, g);
    return;
  }
  // scale gradient and objective sums: loss block t in thread t, pairwise tree
  for (int c = 0; c < 4; ++c)
    for (int t = tid; t < kTdesMaxLossBlocks; t += kUpdThreads)
      tree[c][t] = t < u.loss_blocks ? u.part_d[t * 4 + c] : 0.0;
  __syncthreads();
  for (int half = kTdesMaxLossBlocks / 2; half > 0; half >>= 1) {
    for (int t = tid; t < 4 * half; t += kUpdThreads) tree[t / half][t % half] += tree[t / half][t % half + half];
    __syncthreads();
  }
  if (tid != 0) return;
  adamw(u, u.n_params - 1, tree[0][0]);
  if (u.loss) {
    const double kl = u.G ? tree[1][0] / u.G : 0.0;
    const double pr = u.P ? tree[2][0] / u.P : 0.0;
    const double bce = u.G ? tree[3][0] / (static_cast<double>(u.G) * u.K) : 0.0;
    u.loss[0] = u.lambda_kl * kl + u.lambda_pair * pr + u.lambda_bce * bce;
    u.loss[1] = kl;
    u.loss[2] = pr;
    u.loss[3] = bce;
  }
}

size_t loss_lds_bytes(int E, int M16, int L) {
  return sizeof(float) * (2 * static_cast<size_t>(E) * (M16 + 4) + static_cast<size_t>(L) * M16 +
                          static_cast<size_t>(kLossWaves) * L * M16 + kLossWaves * 3 * kMaxK) +
         sizeof(double) * kLossWaves * 4;
}

template <int NT, int EB>
bool launch_t(const TrainArgs &a, int nt, int eb, int loss_blocks, int child_blocks,
              int grad_blocks, hipStream_t stream) {
  if (nt != NT || eb != EB) return false;
  const size_t lds = loss_lds_bytes(EB * 16, NT * 16, a.L);
  // child tiles of 16 rows per group: K <= 16, 32 or 64
  if (a.K <= 16)
    hipLaunchKernelGGL((loss_kernel<NT, EB, 1>), dim3(loss_blocks), dim3(kLossThreads), lds, stream, a);
  else if (a.K <= 32)
    hipLaunchKernelGGL((loss_kernel<NT, EB, 2>), dim3(loss_blocks), dim3(kLossThreads), lds, stream, a);
  else
    hipLaunchKernelGGL((loss_kernel<NT, EB, 4>), dim3(loss_blocks), dim3(kLossThreads), lds, stream, a);
  if (grad_blocks > 0)
    hipLaunchKernelGGL((wgrad_kernel<NT, EB>), dim3(grad_blocks), dim3(kGradThreads), 0, stream, a,
                       child_blocks);
  return true;
}

// the instantiated shapes: E in {32, 64, 128} with E * M16 <= 4096
bool dispatch(const TrainArgs &a, int nt, int eb, int lb, int cb, int gb, hipStream_t st) {
  return launch_t<1, 2>(a, nt, eb, lb, cb, gb, st) || launch_t<1, 4>(a, nt, eb, lb, cb, gb, st) ||
         launch_t<1, 8>(a, nt, eb, lb, cb, gb, st) || launch_t<2, 2>(a, nt, eb, lb, cb, gb, st) ||
         launch_t<2, 4>(a, nt, eb, lb, cb, gb, st) || launch_t<2, 8>(a, nt, eb, lb, cb, gb, st) ||
         launch_t<3, 2>(a, nt, eb, lb, cb, gb, st) || launch_t<3, 4>(a, nt, eb, lb, cb, gb, st) ||
         launch_t<4, 2>(a, nt, eb, lb, cb, gb, st) || launch_t<4, 4>(a, nt, eb, lb, cb, gb, st);
}

}  // namespace

TdesPlan tdes_plan(const graft_tdes_dims &d, int G, int P) {
  TdesPlan p;
  const int64_t items = static_cast<int64_t>(G) + (static_cast<int64_t>(P) + 7) / 8;
  const int64_t lb = (items + 2 * kLossWaves - 1) / (2 * kLossWaves);   // about 2 items per wave
  p.loss_blocks = static_cast<int>(lb < 1 ? 1 : lb > kTdesMaxLossBlocks ? kTdesMaxLossBlocks : lb);
  const int64_t rc = static_cast<int64_t>(G) * d.top_k + 2 * static_cast<int64_t>(P);
  const int64_t rp = static_cast<int64_t>(G) + 2 * static_cast<int64_t>(P);
  p.child_blocks = static_cast<int>((rc + kGradRows - 1) / kGradRows);
  p.parent_blocks = static_cast<int>((rp + kGradRows - 1) / kGradRows);
  return p;
}

TdesWorkspace tdes_workspace(const graft_tdes_dims &d) {
  const TdesPlan most = tdes_plan(d, d.max_groups, d.max_pairs);
  const int64_t m16 = (d.score_dim + 15) / 16 * 16;
  TdesWorkspace w;
  w.dyc = (static_cast<int64_t>(d.max_groups) * d.top_k + 2 * static_cast<int64_t>(d.max_pairs)) * m16;
  w.dyp = (static_cast<int64_t>(d.max_groups) + 2 * static_cast<int64_t>(d.max_pairs)) * m16;
  w.part_u = chunked_size(d.num_pos * d.score_dim, kTdesMaxLossBlocks);
  w.part_d = 4 * static_cast<int64_t>(kTdesMaxLossBlocks);
  w.part_w = chunked_size(d.emb_dim * d.score_dim, most.child_blocks) +
             chunked_size(d.emb_dim * d.score_dim, most.parent_blocks);
  return w;
}

bool tdes_shape_supported(int E, int m, int L, int K) {
  const int m16 = (m + 15) / 16 * 16;
  const bool e_ok = E == 32 || E == 64 || E == 128;
  return e_ok && m >= 1 && m <= kMaxScoreDim && E * m16 <= kMaxEM && L >= 1 && L * m16 <= kMaxLM &&
         K >= 1 && K <= kMaxK && loss_lds_bytes(E, m16, L) <= 64 * 1024;
}

hipError_t launch_tdes_step(graft_tdes *t, const float *emb, const graft_tdes_batch *b,
                            const graft_tdes_hyper *h, int32_t step, float *theta, float *m1,
                            float *m2, double *loss, float *grad, hipStream_t stream) {
  const graft_tdes_dims &d = t->dims;
  const int E = d.emb_dim, m = d.score_dim, L = d.num_pos, K = d.top_k;
  const int G = b->n_groups, P = b->n_pairs;
  const TdesPlan plan = tdes_plan(d, G, P);
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
  a.dyc = t->dyc;
  a.dyp = t->dyp;
  a.part_u = t->part_u;
  a.part_d = t->part_d;
  a.part_w = t->part_w;
  a.error_flag = t->error_flag;
  const int grad_blocks = plan.child_blocks + plan.parent_blocks;
  if (!dispatch(a, (m + 15) / 16, E / 16, plan.loss_blocks, plan.child_blocks, grad_blocks, stream))
    return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  UpdateArgs u;
  u.theta = theta;
  u.m1 = m1;
  u.m2 = m2;
  u.grad_out = grad;
  u.part_u = t->part_u;
  u.part_w = t->part_w;
  u.part_d = t->part_d;
  u.loss = loss;
  u.E = E;
  u.m = m;
  u.L = L;
  u.n_params = 2 * E * m + L * m + 1;
  u.loss_blocks = plan.loss_blocks;
  u.child_blocks = plan.child_blocks;
  u.parent_blocks = plan.parent_blocks;
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
  const int blocks = 2 * ((E * m + kChunk - 1) / kChunk) + (L * m + kChunk - 1) / kChunk + 1;
  hipLaunchKernelGGL(update_kernel, dim3(blocks), dim3(kUpdThreads), 0, stream, u);
  return hipGetLastError();
}

}  // namespace graft
