// k_verify.hip -- verifier-side consumers of a round (the step after emission
// and acceptance; the paper's Preliminaries: the target model verifies the
// tree under a tree-attention mask and commits the longest accepted path).
//
// bias_kernel: expands the ancestor bitset of every node into its row of the
//   draft block's additive attention bias (0 where the node may attend, -inf
//   elsewhere).  One wave per row; each lane writes 16-byte chunks (8 bf16 or
//   4 fp32 entries) from one 64-bit mask word it holds.  Write-bound: the
//   bias is the only large stream.
// commit_kernel: moves the key/value rows of the accepted nodes to
//   consecutive rows.  One workgroup per (plane, sequence, 4 KiB column chunk
//   of a row); each thread owns 16 bytes of the chunk and loads them from up
//   to 16 accepted rows before storing any, so a compaction in place never
//   overwrites a row it has still to read (accepted node indices increase
//   along the path and are >= their position).
#include "graft_internal.h"

namespace graft {
namespace {

constexpr int kBiasWaves = 4;
constexpr int kCommitThreads = 256;
constexpr int kCommitGroup = 16;   // accepted rows loaded before any store

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <bool BF16>
__global__ void __launch_bounds__(kBiasWaves * kWave)
bias_kernel(int batch, int n_max, int words, const int32_t *__restrict__ n_nodes,
            const uint64_t *__restrict__ mask, void *__restrict__ bias, int64_t ld,
            int64_t batch_stride) {
  const int lane = lane_id();
  const int64_t row_id = static_cast<int64_t>(blockIdx.x) * kBiasWaves + threadIdx.x / kWave;
  if (row_id >= static_cast<int64_t>(batch) * n_max) return;
  const int b = static_cast<int>(row_id / n_max), i = static_cast<int>(row_id % n_max);
  int n = n_nodes[b];
  n = n < 0 ? 0 : (n > n_max ? n_max : n);
  const uint64_t *mrow = mask + (static_cast<int64_t>(b) * n_max + i) * words;
  constexpr int kPer = BF16 ? 8 : 4;                 // entries per 16-byte chunk
  const int nfull = n_max / kPer;
  char *out = static_cast<char *>(bias) +
              (static_cast<int64_t>(b) * batch_stride + static_cast<int64_t>(i) * ld) *
                  (BF16 ? 2 : 4);
  for (int c = lane; c * kPer < n_max; c += kWave) {
    const int j0 = c * kPer;
    const uint64_t word = i < n ? mrow[j0 >> 6] : 0ull;
    const uint32_t bits = static_cast<uint32_t>(word >> (j0 & 63)) & ((1u << kPer) - 1u);
    uint32_t v[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const bool vis = ((bits >> k) & 1u) && j0 + k < n;
      v[k] = vis ? 0u : (BF16 ? 0xFF80u : 0xFF800000u);
    }
    if (c < nfull) {
      u32x4 q;
      if (BF16) {
        q = u32x4{v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16),
                  v[6] | (v[7] << 16)};
      } else {
        q = u32x4{v[0], v[1], v[2], v[3]};
      }
      *reinterpret_cast<u32x4 *>(out + static_cast<int64_t>(c) * 16) = q;
    } else {
      // ragged tail of a row whose length is not a multiple of kPer
      for (int k = 0; k < kPer && j0 + k < n_max; ++k) {
        if (BF16)
          reinterpret_cast<uint16_t *>(out)[j0 + k] = static_cast<uint16_t>(v[k]);
        else
          reinterpret_cast<uint32_t *>(out)[j0 + k] = v[k];
      }
    }
  }
}

__global__ void __launch_bounds__(kCommitThreads)
commit_kernel(int batch, int L, int n_max, int chunks, const int32_t *__restrict__ acc_len,
              const int32_t *__restrict__ acc_nodes, const char *src, char *dst,
              int64_t row_bytes, int64_t sp, int64_t sb, int64_t sr, int64_t dp, int64_t db,
              int64_t dr, uint32_t *__restrict__ error_flag) {
  const int chunk = blockIdx.x % chunks;
  const int pb = blockIdx.x / chunks;
  const int b = pb % batch, p = pb / batch;
  int a = acc_len[b];
  a = a < 0 ? 0 : (a > L ? L : a);
  const int64_t col = (static_cast<int64_t>(chunk) * kCommitThreads + threadIdx.x) * 16;
  const bool active = col < row_bytes;
  const char *s0 = src + p * sp + b * sb + col;
  char *d0 = dst + p * dp + b * db + col;
  const int32_t *nodes = acc_nodes + static_cast<int64_t>(b) * L;
  for (int g = 0; g < a; g += kCommitGroup) {
    u32x4 v[kCommitGroup];
    bool ok[kCommitGroup];
#pragma unroll
    for (int k = 0; k < kCommitGroup; ++k) {
      const int i = g + k;
      ok[k] = false;
      if (i < a) {
        const int r = nodes[i];
        ok[k] = r >= 0 && r < n_max;
        if (!ok[k] && threadIdx.x == 0 && chunk == 0) atomicOr(error_flag, 4u);
        if (ok[k] && active) v[k] = *reinterpret_cast<const u32x4 *>(s0 + r * sr);
      }
    }
#pragma unroll
    for (int k = 0; k < kCommitGroup; ++k)
      if (ok[k] && active) *reinterpret_cast<u32x4 *>(d0 + (g + k) * dr) = v[k];
  }
}

}  // namespace

hipError_t launch_mask_to_bias(graft_ctx *ctx, int batch, const int32_t *n_nodes,
                               const uint64_t *mask, void *bias, int dtype, int64_t ld,
                               int64_t batch_stride, hipStream_t stream) {
  const int n_max = ctx->dims.max_nodes, words = (n_max + 63) / 64;
  const int64_t rows = static_cast<int64_t>(batch) * n_max;
  const dim3 grid(static_cast<unsigned>((rows + kBiasWaves - 1) / kBiasWaves));
  if (dtype == 1)
    hipLaunchKernelGGL(bias_kernel<true>, grid, dim3(kBiasWaves * kWave), 0, stream, batch,
                       n_max, words, n_nodes, mask, bias, ld, batch_stride);
  else
    hipLaunchKernelGGL(bias_kernel<false>, grid, dim3(kBiasWaves * kWave), 0, stream, batch,
                       n_max, words, n_nodes, mask, bias, ld, batch_stride);
  return hipGetLastError();
}

hipError_t launch_commit(graft_ctx *ctx, int batch, const int32_t *acc_len,
                         const int32_t *acc_nodes, const void *src, void *dst, int64_t row_bytes,
                         int n_planes, int64_t sp, int64_t sb, int64_t sr, int64_t dp,
                         int64_t db, int64_t dr, hipStream_t stream) {
  const int64_t per = static_cast<int64_t>(kCommitThreads) * 16;
  const int chunks = static_cast<int>((row_bytes + per - 1) / per);
  const int64_t blocks = static_cast<int64_t>(n_planes) * batch * chunks;
  hipLaunchKernelGGL(commit_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kCommitThreads), 0,
                     stream, batch, ctx->dims.num_pos, ctx->dims.max_nodes, chunks, acc_len,
                     acc_nodes, static_cast<const char *>(src), static_cast<char *>(dst),
                     row_bytes, sp, sb, sr, dp, db, dr, ctx->error_flag);
  return hipGetLastError();
}

}  // namespace graft
