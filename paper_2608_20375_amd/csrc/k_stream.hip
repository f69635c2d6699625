// k_stream.hip -- a plain read of a device buffer: the HBM read rate that a
// streaming kernel can reach on this GPU, measured next to the logits pass
// (which reads its bf16 rows with the same 16-byte non-temporal loads).
//
// read_stream_kernel: 2048 workgroups of 256 lanes stride over the 16-byte
// vectors, one load per lane per step (measured faster than 2 to 8 loads in
// flight per lane, than contiguous chunks per workgroup, than 4096 or 8192
// workgroups, and than cached loads); every word is folded into an xor so
// that the loads stay live, the lanes of a block combine theirs, and block i
// writes sink[i].  Block 0 zeroes
// the sink words past the grid, so the xor of all kReadSinkWords sink words is
// the xor of every 32-bit word of the buffer.
#include "graft_internal.h"

static_assert(2048 <= graft::kReadSinkWords, "one sink word per workgroup");

namespace graft {
namespace {

constexpr int kStreamThreads = 256;
constexpr int kStreamWaves = kStreamThreads / kWave;
constexpr int kStreamBlocks = 2048;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t fold(u32x4 v) { return (v.x ^ v.y) ^ (v.z ^ v.w); }

__global__ void __launch_bounds__(kStreamThreads)
read_stream_kernel(const u32x4 *__restrict__ p, int64_t n, uint32_t *__restrict__ sink) {
  __shared__ uint32_t s_x[kStreamWaves];
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kStreamThreads;
  int64_t i = static_cast<int64_t>(blockIdx.x) * kStreamThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i < n; i += stride) acc ^= fold(__builtin_nontemporal_load(p + i));
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) acc ^= xor_lane(acc, o);
  const int wave = threadIdx.x / kWave;
  if (lane_id() == 0) s_x[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t x = 0;
    for (int w = 0; w < kStreamWaves; ++w) x ^= s_x[w];
    sink[blockIdx.x] = x;
  }
  if (blockIdx.x == 0)
    for (int k = gridDim.x + threadIdx.x; k < kReadSinkWords; k += kStreamThreads) sink[k] = 0u;
}

}  // namespace

hipError_t launch_read_stream(const void *src, int64_t bytes, uint32_t *sink, hipStream_t stream) {
  const int64_t n = bytes / 16;
  int64_t blocks = (n + kStreamThreads - 1) / kStreamThreads;
  if (blocks > kStreamBlocks) blocks = kStreamBlocks;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(read_stream_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kStreamThreads),
                     0, stream, static_cast<const u32x4 *>(src), n, sink);
  return hipGetLastError();
}

}  // namespace graft
