// Tail-entropy block scores, start-block choice and refresh flags, gfx950.
//
// Paper, Sec. "Training-Free MBE Decoding", paragraph on tail-entropy block
// selection, Eqs. (5)-(6): a block's score is the mean of its ceil(rho B)
// largest per-position entropies; the editing window of block j starts at the
// best-scoring block among the K_max - 1 blocks before j.  Sec.
// "Infrastructure Optimization", cache control: after editing, the blocks that
// changed are recomputed (refresh flags).
//
// These are small per-block or per-sequence reductions; each runs as one
// launch with no workspace.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mbe {
namespace {

constexpr int kMaxBlock = 1024;   // rows per block the score kernel sorts in LDS

// One workgroup per block: the entropies are sorted in LDS (bitonic, largest
// first, padded with -inf to a power of two) and thread 0 sums the first k
// in order, so the result does not depend on the launch shape.
__global__ __launch_bounds__(256) void tail_entropy_kernel(const float *entropy, int32_t block_size, int32_t k,
                                                           float *scores) {
  __shared__ float v[kMaxBlock];
  const int64_t blk = blockIdx.x;
  int n = 1;
  while (n < block_size) n <<= 1;
  for (int i = threadIdx.x; i < n; i += 256) v[i] = i < block_size ? entropy[blk * block_size + i] : -INFINITY;
  __syncthreads();
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < n; i += 256) {
        const int j = i ^ stride;
        if (j > i) {
          const bool desc = (i & size) == 0;   // descending runs first: the final order is descending
          const float a = v[i], b = v[j];
          if (desc ? (a < b) : (a > b)) {
            v[i] = b;
            v[j] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) {
    float sum = 0.f;
    for (int i = 0; i < k; ++i) sum += v[i];
    scores[blk] = sum / static_cast<float>(k);
  }
}

// One thread per sequence: argmax over the candidate blocks, earliest on ties.
__global__ __launch_bounds__(256) void select_start_kernel(const float *scores, int32_t batch, int32_t stride,
                                                           const int32_t *current, int32_t k_max, int32_t *start) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= batch) return;
  const int j = min(max(current[b], 0), stride);
  int best = j;
  float best_s = 0.f;
  for (int i = max(0, j - k_max + 1); i < j; ++i) {
    const float s = scores[static_cast<int64_t>(b) * stride + i];
    if (best == j || s > best_s) {
      best = i;
      best_s = s;
    }
  }
  start[b] = best;
}

// One thread per sequence: changed blocks, and in the second mode every block
// after the first changed one.
__global__ __launch_bounds__(256) void refresh_kernel(const uint8_t *changed, int32_t batch, int32_t num_blocks,
                                                      int32_t mode, uint8_t *refresh) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= batch) return;
  bool seen = false;
  for (int i = 0; i < num_blocks; ++i) {
    const int64_t at = static_cast<int64_t>(b) * num_blocks + i;
    const bool c = changed[at] != 0;
    seen |= c;
    refresh[at] = (c || (seen && mode == 1)) ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_tail_entropy_scores(const float *entropy, int64_t num_blocks, int32_t block_size, int32_t k,
                                      float *scores, hipStream_t stream) {
  hipLaunchKernelGGL(tail_entropy_kernel, dim3(static_cast<unsigned>(num_blocks)), dim3(256), 0, stream, entropy,
                     block_size, k, scores);
  return hipGetLastError();
}

hipError_t launch_select_start_block(const float *scores, int32_t batch, int32_t stride, const int32_t *current,
                                     int32_t k_max, int32_t *start, hipStream_t stream) {
  hipLaunchKernelGGL(select_start_kernel, dim3(static_cast<unsigned>((batch + 255) / 256)), dim3(256), 0, stream,
                     scores, batch, stride, current, k_max, start);
  return hipGetLastError();
}

hipError_t launch_refresh_blocks(const uint8_t *changed, int32_t batch, int32_t num_blocks, int32_t mode,
                                 uint8_t *refresh, hipStream_t stream) {
  hipLaunchKernelGGL(refresh_kernel, dim3(static_cast<unsigned>((batch + 255) / 256)), dim3(256), 0, stream, changed,
                     batch, num_blocks, mode, refresh);
  return hipGetLastError();
}

}  // namespace mbe
