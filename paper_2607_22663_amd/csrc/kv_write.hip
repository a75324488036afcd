// Write-back of recomputed K/V into the paged pools, gfx950.
//
// Paper, Sec. "Infrastructure Optimization", cache control: the editing pass
// leaves the cache untouched; afterwards the changed blocks are recomputed
// under standard attention and their K/V written back.  This kernel is that
// write: token t of sequence b goes to absolute position start_b + t, i.e.
// slot (position % 16) of page page_table[b][position / 16].  With block
// flags only the tokens of flagged blocks (block t / B of the write) are
// written: the blocks the refresh recomputed.
//
// One workgroup per (sequence, page touched, KV head).  The workgroup first
// decides which of the page's 16 slots it writes (in range, a row of the
// input, a flagged block), then copies K rows (and V rows of a token-major
// pool) as 16-byte chunks.  For a token-minor V pool ([D][16] per page and
// head) the workgroup stages its tokens' V rows in LDS, then writes each
// dim's run of slots, 16 bytes at a time where all 8 slots of a half-row are
// written.  A table slot past the
// row or a page id outside the pool writes nothing.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mbe {
namespace {

__global__ __launch_bounds__(256) void kv_write_kernel(KvWriteParams p) {
  __shared__ __align__(16) uint16_t vs[kPageSize * 128];   // [slot][D], D <= 128
  const int b = blockIdx.y;
  const int g = blockIdx.z;
  const int D = p.head_dim;
  const int len = min(max(p.lens[b], 0), p.max_len);
  if (len == 0) return;
  const int start = max(p.start_pos[b], 0);
  const int page_slot = start / kPageSize + static_cast<int>(blockIdx.x);   // page index within the row
  const int p0 = max(start, page_slot * kPageSize);                          // positions [p0, p1) on this page
  const int p1 = min(start + len, (page_slot + 1) * kPageSize);
  if (p0 >= p1 || page_slot >= p.max_pages) return;
  const int32_t pid = p.page_table[static_cast<int64_t>(b) * p.max_pages + page_slot];
  if (pid < 0 || pid >= p.num_pages) return;
  // first row of sequence b: the lengths before it, summed across the lanes
  // of the wave (independent loads, then a butterfly)
  int64_t row0 = 0;
  for (int j = threadIdx.x & 63; j < b; j += 64) row0 += min(max(p.lens[j], 0), p.max_len);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) row0 += __shfl_xor(row0, o);
  // slots of this page that are written: bit s for slot s (same in every lane)
  uint32_t wmask = 0;
  for (int pos = p0; pos < p1; ++pos) {
    const int t = pos - start;
    const bool in_rows = row0 + t < p.total_tokens;
    const bool flagged = !p.block_flags || p.block_flags[static_cast<int64_t>(b) * p.flag_stride + t / p.block_size];
    if (in_rows && flagged) wmask |= 1u << (pos % kPageSize);
  }
  if (wmask == 0) return;
  const int64_t page_base = (static_cast<int64_t>(pid) * p.num_kv_heads + g) * kPageSize * D;   // elements
  const int chunks = D / 8;
  const int n = p1 - p0;
  // K: [slot][D], a 16-byte chunk per thread.  V: the same when the pool is
  // token-major; otherwise its rows are staged in LDS as [slot][D]
  for (int i = threadIdx.x; i < n * chunks; i += 256) {
    const int tok = i / chunks, c = i % chunks;
    const int slot = (p0 + tok) % kPageSize;
    if (!((wmask >> slot) & 1u)) continue;
    const int64_t row = row0 + (p0 - start) + tok;
    const uint4 wk = *reinterpret_cast<const uint4 *>(p.k_new + (row * p.num_kv_heads + g) * D + c * 8);
    const uint4 wv = *reinterpret_cast<const uint4 *>(p.v_new + (row * p.num_kv_heads + g) * D + c * 8);
    *reinterpret_cast<uint4 *>(p.k_pages + page_base + slot * D + c * 8) = wk;
    if (p.v_token_major) *reinterpret_cast<uint4 *>(p.v_pages + page_base + slot * D + c * 8) = wv;
    else *reinterpret_cast<uint4 *>(vs + slot * D + c * 8) = wv;
  }
  if (p.v_token_major) return;
  __syncthreads();
  // V: [D][slot], per (dim, half of 8 slots)
  for (int i = threadIdx.x; i < D * 2; i += 256) {
    const int d = i >> 1, h = i & 1;
    const int a = h * 8;
    const uint32_t half = (wmask >> a) & 0xFFu;
    if (half == 0) continue;
    uint16_t *dst = p.v_pages + page_base + static_cast<int64_t>(d) * kPageSize + a;
    if (half == 0xFFu) {
      uint4 w;
      uint32_t *u = reinterpret_cast<uint32_t *>(&w);
#pragma unroll
      for (int k = 0; k < 4; ++k)
        u[k] = static_cast<uint32_t>(vs[(a + 2 * k) * D + d]) | (static_cast<uint32_t>(vs[(a + 2 * k + 1) * D + d]) << 16);
      *reinterpret_cast<uint4 *>(dst) = w;
    } else {
      for (int s = 0; s < 8; ++s)
        if ((half >> s) & 1u) dst[s] = vs[(a + s) * D + d];
    }
  }
}

}  // namespace

hipError_t launch_kv_write(const KvWriteParams &p, hipStream_t stream) {
  // pages a sequence's range can touch: ceil(max_len / 16) + 1 (an unaligned start)
  const unsigned pages = static_cast<unsigned>((p.max_len + kPageSize - 1) / kPageSize + 1);
  hipLaunchKernelGGL(kv_write_kernel, dim3(pages, static_cast<unsigned>(p.batch), static_cast<unsigned>(p.num_kv_heads)),
                     dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace mbe
