// edge_mfma.h -- the TDES edge scores of one (sequence, depth) by one wave
// (eqs. tdes-bitower, tdes-center, tdes-score).  Shared by the edge stage and
// by the selection kernel's fused path, so that both produce the same bits.
//
// Inputs (LDS): the n_par parent rows g_p + u_d and the K child rows g_c + u_d
// (m floats each, rows ld floats apart, ld % 4 == 0 and 16-byte aligned
// rows), log q and the token-id rank (column) of each child, and the rank
// (row) of each parent (prank == nullptr: row 0).  Per parent p and child c:
//   f = scale * <par[p], chd[c]> / sqrt(m),  S = log q(c) + beta * (f - mean_c f)
// (the mean over the K children when center != 0), stored at
// rows[prank[p] * K + col[c]] (selection's token-id order) and, when out is
// given, at out[p * K + c] (rank order).  Both return this lane's "some stored
// S > 0"; the whole wave must call them.
//   edge_tiles (m a multiple of 16): the n_par x K products on fp32 matrix
//     cores, 16 x 16 tiles of v_mfma_f32_16x16x4f32;
//   edge_passes (other m): VALU dot products, SEG lanes per parent.
#pragma once

#include "graft_internal.h"

namespace graft {

typedef float mfma_f32x4 __attribute__((ext_vector_type(4)));

// Sum over the 16 lanes of each row of the wave (lanes 16 g .. 16 g + 15), in
// every lane of the row: butterfly steps 1, 2, 4, 8.
__device__ __forceinline__ float row16_sum(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __uint_as_float(xor_lane(__float_as_uint(v), o));
  return v;
}

// One (sequence, depth) for edge_tiles: its parent and child rows, number of
// parents, log q and column of each child, row of each parent (prank ==
// nullptr: 0), and the outputs.
struct EdgeJob {
  const float *par, *chd;
  int n_par;
  const float *lq;
  const int32_t *col, *prank;
  float *rows, *out;
};

// Matrix-core tiles for ND jobs of the same K, interleaved (independent
// accumulator chains; each job's arithmetic is the same as alone).  Lane
// (i = lane % 16, g = lane / 16) feeds parent row 16 tp + i and child row
// 16 tc + i at k = g * MK + t (t < MK, m = 4 MK: two or more 16-byte loads per
// row) and receives f of parents 16 tp + 4 g + r (r < 4) with child 16 tc + i.
// NT >= ceil(K / 16) column tiles (those past K hold zeros); a parent's mean
// sums each column tile's row (row16_sum), combines the tiles as
// (t0 + t1) + (t2 + t3) and scales by fl(1 / K).
template <int MK, int NT, int ND>
__device__ __forceinline__ bool edge_tiles(const EdgeJob (&job)[ND], int ld, int K, float fscale,
                                           float beta, int center) {
  static_assert(MK % 4 == 0 && (NT == 1 || NT == 2 || NT == 4), "tile shape");
  constexpr int V4 = MK / 4;
  const int lane = lane_id(), i = lane & 15, g = lane >> 4;
  // the children's operands of every column tile, kept across parent tiles
  float4 bv[ND][NT][V4];
  float lqv[ND][NT];
  int32_t colv[ND][NT];
  int n_tp = 0;
#pragma unroll
  for (int d = 0; d < ND; ++d) {
    const int nt = (job[d].n_par + 15) >> 4;
    n_tp = nt > n_tp ? nt : n_tp;
#pragma unroll
    for (int tc = 0; tc < NT; ++tc) {
      const int c = tc * 16 + i;
      const int cc = c < K ? c : 0;
      const float4 *src = reinterpret_cast<const float4 *>(job[d].chd + cc * ld + g * MK);
#pragma unroll
      for (int t = 0; t < V4; ++t) bv[d][tc][t] = src[t];
      lqv[d][tc] = job[d].lq[cc];
      colv[d][tc] = job[d].col[cc];
    }
  }
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int tc = 0; tc < NT; ++tc)
      if (tc * 16 + i >= K)
#pragma unroll
        for (int t = 0; t < V4; ++t) bv[d][tc][t] = make_float4(0.f, 0.f, 0.f, 0.f);
  const float inv_k = 1.0f / static_cast<float>(K);
  bool pos = false;
  for (int tp = 0; tp < n_tp; ++tp) {
    const int pa = tp * 16 + i;
    float4 av[ND][V4];
    int32_t prow[ND][4];
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      const int np = job[d].n_par;
      const float4 *src =
          reinterpret_cast<const float4 *>(job[d].par + (pa < np ? pa : 0) * ld + g * MK);
#pragma unroll
      for (int t = 0; t < V4; ++t) av[d][t] = src[t];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int p = tp * 16 + 4 * g + r;
        prow[d][r] = job[d].prank ? job[d].prank[p < np ? p : 0] : 0;
      }
    }
#pragma unroll
    for (int d = 0; d < ND; ++d)
      if (pa >= job[d].n_par)
#pragma unroll
        for (int t = 0; t < V4; ++t) av[d][t] = make_float4(0.f, 0.f, 0.f, 0.f);
    mfma_f32x4 acc[ND][NT];
#pragma unroll
    for (int tc = 0; tc < NT; ++tc)
#pragma unroll
      for (int d = 0; d < ND; ++d) acc[d][tc] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < V4; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int tc = 0; tc < NT; ++tc)
#pragma unroll
          for (int d = 0; d < ND; ++d)
            acc[d][tc] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[d][t][q], bv[d][tc][t][q],
                                                               acc[d][tc], 0, 0, 0);
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      if (tp * 16 >= job[d].n_par) continue;   // this job has no parent tile tp
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int p = tp * 16 + 4 * g + r;
        const bool pok = p < job[d].n_par;
        float f[NT];
#pragma unroll
        for (int tc = 0; tc < NT; ++tc) f[tc] = fscale * acc[d][tc][r];
        float mean = 0.f;
        if (center) {
          float rs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int tc = 0; tc < NT; ++tc) rs[tc] = row16_sum(tc * 16 + i < K ? f[tc] : 0.f);
          mean = ((rs[0] + rs[1]) + (rs[2] + rs[3])) * inv_k;
        }
#pragma unroll
        for (int tc = 0; tc < NT; ++tc) {
          const int c = tc * 16 + i;
          const bool valid = pok && c < K;
          const float S = (lqv[d][tc] + beta * (f[tc] - mean)) + 0.0f;   // -0 -> +0
          if (valid) {
            job[d].rows[prow[d][r] * K + colv[d][tc]] = S;
            if (job[d].out) job[d].out[p * K + c] = S;
          }
          pos |= valid && S > 0.f;
        }
      }
    }
  }
  return pos;
}

// Sum over each run of seg consecutive lanes (seg a power of two), in every
// lane of the run: butterfly steps 1, 2, ... seg / 2.
__device__ __forceinline__ float seg_sum_rt(float v, int seg) {
#pragma unroll
  for (int stride = 1; stride < kWave; stride <<= 1)
    if (stride < seg) v += __uint_as_float(xor_lane(__float_as_uint(v), stride));
  return v;
}

// VALU passes: SEG lanes per parent (SEG = K rounded up to a power of two),
// 64 / SEG parents a pass; lane c of a run keeps child c's row in registers
// (KQ >= ceil(m / 4) groups of four; with m % 4 != 0 one float at a time)
// and reads the parent's row from LDS (one address for the whole run).
template <int KQ>
__device__ __forceinline__ bool edge_passes(const float *par, const float *chd, int ld, int n_par,
                                            int K, int m, float fscale, float beta, int center,
                                            const float *lq, const int32_t *col,
                                            const int32_t *prank, float *rows, float *out) {
  const int lane = lane_id();
  int seg = 1;
  while (seg < K) seg <<= 1;
  const int kRows = kWave / seg;
  const int c = lane & (seg - 1), cc = c < K ? c : 0;
  const int m4 = (m & 3) == 0 ? m >> 2 : 0;
  float4 cr[KQ];
  if (m4 > 0) {
    const float4 *c4 = reinterpret_cast<const float4 *>(chd + cc * ld);
#pragma unroll
    for (int q = 0; q < KQ; ++q) cr[q] = c4[q < m4 ? q : 0];
#pragma unroll
    for (int q = 0; q < KQ; ++q)
      if (q >= m4) cr[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const float lqc = lq[cc];
  const int colc = col[cc];
  bool pos = false;
  for (int p0 = 0; p0 < n_par; p0 += kRows) {
    const int p = p0 + lane / seg;
    const bool valid = p < n_par && c < K;
    const int pp = p < n_par ? p : 0;
    const int prow = prank ? prank[pp] : 0;
    const float *pv = par + pp * ld;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    if (m4 > 0) {
      const float4 *p4 = reinterpret_cast<const float4 *>(pv);
      float4 x[KQ];
#pragma unroll
      for (int q = 0; q < KQ; ++q) x[q] = p4[q < m4 ? q : 0];
#pragma unroll
      for (int q = 0; q < KQ; ++q) {
        a0 = __builtin_fmaf(x[q].x, cr[q].x, a0);
        a1 = __builtin_fmaf(x[q].y, cr[q].y, a1);
        a2 = __builtin_fmaf(x[q].z, cr[q].z, a2);
        a3 = __builtin_fmaf(x[q].w, cr[q].w, a3);
      }
    } else {
      const float *cv = chd + cc * ld;
#pragma unroll 4
      for (int j = 0; j < m; ++j) a0 = __builtin_fmaf(pv[j], cv[j], a0);
    }
    const float f = fscale * ((a0 + a1) + (a2 + a3));
    float mean = 0.f;
    if (center) mean = seg_sum_rt(valid ? f : 0.f, seg) / static_cast<float>(K);
    const float S = (lqc + beta * (f - mean)) + 0.0f;   // -0 -> +0
    if (valid) {
      rows[prow * K + colc] = S;
      if (out) out[p * K + c] = S;
    }
    pos |= valid && S > 0.f;
  }
  return pos;
}

}  // namespace graft
