// Editing-window attention over a paged KV prefix, gfx950 (MI355X).
//
// Paper, Sec. "Training-Free MBE Decoding", Eq. (4): after block j converges
// the window W_j = [j*B, (j+1)B) is re-run with full attention inside the
// window, reading the committed prefix from the KV cache without writing it
// (Sec. "Infrastructure Optimization", cache control).  The block-causal mode
// is the standard block-diffusion scope (Sec. "Block diffusion").
//
// Work decomposition
//   All G = Hq/Hkv query heads of a KV head share its keys, so the rows of
//   one (sequence b, KV head g) are packed: row r = i*G + hl is window
//   position i of query head g*G + hl.  A workgroup (4 waves) owns 256 such
//   rows and one split of the key range; a wave owns 64 rows as two 32-row
//   MFMA column blocks.
//
// Contractions on bf16 MFMA (v_mfma_f32_32x32x16_bf16)
//   S^T = K . Q^T : A = 32 keys x 16 dims from LDS, B = Q^T from registers.
//                  The result holds one query per lane (column), so the
//                  softmax row statistics stay in the lane; only the two
//                  32-lane halves, which hold different keys of the same
//                  query, exchange the maximum once per tile.
//   O^T += V^T . P^T : A = 32 dims x 16 keys of V^T from LDS, B = P^T taken
//                  straight from the S^T accumulators.  Keys are assigned to
//                  MFMA rows through a fixed permutation (swap of bits 2 and 3
//                  of the row index) so that the 8 keys a lane contributes to
//                  one P.V step are 8 consecutive keys: with token-minor V
//                  pages that is one 16-byte LDS read per operand.
//
// Softmax: online, base 2, fp32.  The running maximum is only raised when a
// tile exceeds it by more than 2^8 (decided per wave), so the O rescale is
// skipped on most tiles; exponentials stay below 2^8.
//
// Split-KV: long prefixes are cut into kv_chunk-key splits.  Each split
// writes unnormalised O, its maximum and its sum; the last split of a query
// tile to finish (atomic arrival counter, reset after use) merges them in
// split order: M = max m_s, O = sum 2^(m_s-M) O_s / sum 2^(m_s-M) l_s.
//
// K/V tiles of 64 keys (four 16-token pages, gathered through the page table)
// are staged in LDS with a register-prefetch double buffer and padded rows
// (no bank conflicts on the 16-byte operand reads).  Workgroup ids are mapped
// so that each XCD runs a contiguous range of work units and the query tiles
// that share a key range run back to back on the same XCD (shared L2).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mbe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kT = kWaves * 64;
constexpr float kNegInf = -INFINITY;
constexpr float kLazyRescale = 8.0f;   // log2 units

template <int D>
struct Lds {
  static constexpr int kStride = D + 8;          // K row: 64 keys x (D + 8) bf16
  static constexpr int vStride = kKeyTile + 8;   // V^T row: D dims x (64 + 8) bf16
  static constexpr int kElems = kKeyTile * kStride;
  static constexpr int vElems = D * vStride;
  static constexpr int bufElems = kElems + vElems;
  static constexpr int bytes = 2 * bufElems * 2;   // double buffer
};

// Bit swap 2<->3 of a row index in 0..31: MFMA row -> key within a 32-key block.
__device__ __forceinline__ int perm_row(int r) {
  return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to two bf16, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = __builtin_convertvector(f32x2{lo, hi}, bf16x2);
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 lds_read8(const uint16_t *p) {
  return *reinterpret_cast<const bf16x8 *>(p);
}

template <int D>
struct TileLoader {
  // chunks of 8 bf16 (16 bytes): a page holds 2*D chunks of K and 2*D of V
  static constexpr int kChunksPerPage = 2 * D;
  static constexpr int kPagesPerPass = kT / kChunksPerPage;   // 1 (D=128) or 2 (D=64)
  static constexpr int kPasses = (kKeyTile / kPageSize) / kPagesPerPass;
  uint4 k[kPasses];
  uint4 v[kPasses];
  int vvalid[kPasses];      // valid slots of this page for V zero fill (16 = all)

  __device__ __forceinline__ void load(const AttnParams &p, int b, int g, int tile_key0, int n_all) {
    const int tid = threadIdx.x;
    const int c = tid % kChunksPerPage;
#pragma unroll
    for (int j = 0; j < kPasses; ++j) {
      const int pg = j * kPagesPerPass + tid / kChunksPerPage;     // page within tile
      const int tok0 = tile_key0 + pg * kPageSize;
      if (tok0 < n_all) {
        const int slot_in_table = min(tok0 / kPageSize, p.max_pages - 1);
        int page = p.page_table[static_cast<int64_t>(b) * p.max_pages + slot_in_table];
        page = min(max(page, 0), p.num_pages - 1);
        const int64_t base = (static_cast<int64_t>(page) * p.num_kv_heads + g) * (kPageSize * D);
        k[j] = *reinterpret_cast<const uint4 *>(p.k_pages + base + c * 8);
        v[j] = *reinterpret_cast<const uint4 *>(p.v_pages + base + c * 8);
        vvalid[j] = min(kPageSize, n_all - tok0);
      } else {
        k[j] = make_uint4(0, 0, 0, 0);
        v[j] = make_uint4(0, 0, 0, 0);
        vvalid[j] = 0;
      }
    }
  }

  __device__ __forceinline__ void store(uint16_t *buf) const {
    const int tid = threadIdx.x;
    const int c = tid % kChunksPerPage;
    uint16_t *ks = buf;
    uint16_t *vs = buf + Lds<D>::kElems;
#pragma unroll
    for (int j = 0; j < kPasses; ++j) {
      const int pg = j * kPagesPerPass + tid / kChunksPerPage;
      // K page: [16 slots][D]; chunk c = slot * (D/8) + d/8
      const int slot = c / (D / 8);
      const int d0 = (c % (D / 8)) * 8;
      *reinterpret_cast<uint4 *>(ks + (pg * kPageSize + slot) * Lds<D>::kStride + d0) = k[j];
      // V page: [D][16 slots]; chunk c = d * 2 + half
      const int d = c / 2;
      const int s0 = (c % 2) * 8;
      uint4 w = v[j];
      const int nv = vvalid[j] - s0;    // valid slots within this 8-slot chunk
      if (nv < 8) {
        uint32_t *ww = reinterpret_cast<uint32_t *>(&w);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo_keep = (2 * e < nv) ? 0x0000ffffu : 0u;
          const uint32_t hi_keep = (2 * e + 1 < nv) ? 0xffff0000u : 0u;
          ww[e] &= (lo_keep | hi_keep);
        }
      }
      *reinterpret_cast<uint4 *>(vs + d * Lds<D>::vStride + pg * kPageSize + s0) = w;
    }
  }
};

template <int D, int MODE>
__global__ __launch_bounds__(kT, 1) void window_attention_kernel(AttnParams p) {
  __shared__ __align__(16) uint16_t lds[2 * Lds<D>::bufElems];
  __shared__ uint32_t sh_last;

  // ---- work unit: XCD-contiguous ranges of (bg, split, qtile) with qtile fastest
  const int64_t id = blockIdx.x;
  const int64_t w = (id % kXcds) * p.units_per_xcd + id / kXcds;
  if (w >= p.units) return;
  const int qtile = static_cast<int>(w % p.qtiles);
  const int64_t t1 = w / p.qtiles;
  const int split = static_cast<int>(t1 % p.splits);
  const int bg = static_cast<int>(t1 / p.splits);
  const int b = bg / p.num_kv_heads;
  const int g = bg % p.num_kv_heads;

  const int G = p.group;
  // lengths are clamped to the host-validated bounds, so a wrong device value
  // can give wrong numbers but never an access outside q, out or the workspace
  const int P = min(max(p.prefix_lens[b], 0), p.max_prefix);
  const int W = p.fixed_window >= 0 ? p.fixed_window : min(max(p.window_lens[b], 0), p.max_window);
  const int n_all = P + W;
  const int M = G * W;
  const int row0 = qtile * kRowsPerTile;
  if (row0 >= M) return;
  const int nsplit = min(p.splits, max(1, (n_all + p.kv_chunk - 1) / p.kv_chunk));
  if (split >= nsplit) return;
  const int kb = split * p.kv_chunk;
  const int ke = min(n_all, kb + p.kv_chunk);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c = lane & 31;       // query column of this lane
  const int h = lane >> 5;       // which half of the 32x32 MFMA layout

  // first query row of sequence b
  int cu = 0;
  if (p.fixed_window >= 0) {
    cu = b * p.fixed_window;
  } else {
    for (int j = lane; j < b; j += 64) cu += min(max(p.window_lens[j], 0), p.max_window);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cu += __shfl_xor(cu, o);
  }

  // ---- this lane's two query rows (one per 32-row block of the wave)
  int lim[2];
  bool valid[2];
  int64_t qoff[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = row0 + wave * kRowsPerWave + qb * 32 + c;
    valid[qb] = r < M && cu + r / G < p.total_q;
    const int i = valid[qb] ? r / G : 0;
    const int hq = g * G + (valid[qb] ? r % G : 0);
    qoff[qb] = (static_cast<int64_t>(cu + i) * p.num_q_heads + hq) * D;
    int n = n_all;
    if (MODE == 1) n = min(n_all, P + (i / p.block_size + 1) * p.block_size);
    lim[qb] = valid[qb] ? min(n, ke) : ke;
  }
  // keys any row of this workgroup can see
  int kend = ke;
  if (MODE == 1) {
    const int r_last = min(M, row0 + kRowsPerTile) - 1;
    const int i_last = r_last / G;
    kend = min(ke, P + (i_last / p.block_size + 1) * p.block_size);
  }
  const int ntiles = kend > kb ? (kend - kb + kKeyTile - 1) / kKeyTile : 0;
  // smallest limit over the wave: tiles ending at or below it need no mask
  int wmin = min(lim[0], lim[1]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) wmin = min(wmin, __shfl_xor(wmin, o));

  // ---- Q^T operands in registers: lane (c, h) holds dims 16kk + 8h .. +7
  constexpr int KK = D / 16;
  bf16x8 qreg[2][KK];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (valid[qb])
        qreg[qb][kk] = *reinterpret_cast<const bf16x8 *>(p.q + qoff[qb] + kk * 16 + h * 8);
      else
        qreg[qb][kk] = bf16x8{};
    }

  constexpr int DB = D / 32;
  f32x16 acc_o[2][DB];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < DB; ++db) acc_o[qb][db] = f32x16{};
  float m_run[2] = {kNegInf, kNegInf};   // log2 units
  float l_run[2] = {0.f, 0.f};

  // key offset (within a 32-key block) held in accumulator register v
  // of this lane: 16*(v>>3) + 8h + (v&7)
  const int prow = perm_row(c);

  TileLoader<D> ld;
  if (ntiles > 0) {
    ld.load(p, b, g, kb, n_all);
    ld.store(lds);
  }
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const uint16_t *buf = lds + (t & 1) * Lds<D>::bufElems;
    const uint16_t *ks = buf;
    const uint16_t *vs = buf + Lds<D>::kElems;
    const int key0 = kb + t * kKeyTile;
    const bool more = t + 1 < ntiles;
    if (more) ld.load(p, b, g, key0 + kKeyTile, n_all);

    // S^T = K . Q^T for two 32-key blocks x two 32-query blocks
    f32x16 s[2][2];
#pragma unroll
    for (int kbk = 0; kbk < 2; ++kbk) {
      s[kbk][0] = f32x16{};
      s[kbk][1] = f32x16{};
      const uint16_t *krow = ks + (kbk * 32 + prow) * Lds<D>::kStride + h * 8;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8 a = lds_read8(krow + kk * 16);
        s[kbk][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[0][kk], s[kbk][0], 0, 0, 0);
        s[kbk][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[1][kk], s[kbk][1], 0, 0, 0);
      }
    }

    // mask (only on tiles that reach past some row's limit)
    if (key0 + kKeyTile > wmin) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int kbk = 0; kbk < 2; ++kbk)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = key0 + kbk * 32 + 16 * (v >> 3) + 8 * h + (v & 7);
            if (key >= lim[qb]) s[kbk][qb][v] = kNegInf;
          }
    }

    // online softmax; P^T packed to bf16 in MFMA-B layout
    uint32_t pk[2][2][2][4];    // [qb][kbk][m][4 dwords = 8 bf16]
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float mx = kNegInf;
#pragma unroll
      for (int kbk = 0; kbk < 2; ++kbk)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kbk][qb][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mt = mx * p.scale_log2;
      const bool need = mt > m_run[qb] + kLazyRescale;
      if (__any(need)) {
        const float mnew = fmaxf(m_run[qb], mt);
        const float alpha = (mnew == kNegInf) ? 1.f : __builtin_amdgcn_exp2f(m_run[qb] - mnew);
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc_o[qb][db] *= alpha;
        m_run[qb] = mnew;
      }
      const float msafe = (m_run[qb] == kNegInf) ? 0.f : m_run[qb];
      float lsum = 0.f;
#pragma unroll
      for (int kbk = 0; kbk < 2; ++kbk) {
        float e[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          e[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kbk][qb][v], p.scale_log2, -msafe));
          lsum += e[v];
        }
#pragma unroll
        for (int mm = 0; mm < 2; ++mm)
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4)
            pk[qb][kbk][mm][q4] = pack_bf16x2(e[8 * mm + 2 * q4], e[8 * mm + 2 * q4 + 1]);
      }
      l_run[qb] += lsum;
    }

    // O^T += V^T . P^T
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint16_t *vrow = vs + (db * 32 + c) * Lds<D>::vStride + h * 8;
#pragma unroll
      for (int kbk = 0; kbk < 2; ++kbk)
#pragma unroll
        for (int mm = 0; mm < 2; ++mm) {
          const bf16x8 a = lds_read8(vrow + kbk * 32 + mm * 16);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            const bf16x8 bq = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(pk[qb][kbk][mm]));
            acc_o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq, acc_o[qb][db], 0, 0, 0);
          }
        }
    }

    if (more) ld.store(lds + ((t + 1) & 1) * Lds<D>::bufElems);
    __syncthreads();
  }

  // ---- epilogue
  float l_tot[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) l_tot[qb] = l_run[qb] + __shfl_xor(l_run[qb], 32);

  if (nsplit == 1) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      if (!valid[qb]) continue;
      const float inv = l_tot[qb] > 0.f ? 1.f / l_tot[qb] : 0.f;
      uint16_t *orow = p.out + qoff[qb];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int gi = 0; gi < 4; ++gi) {
          const int d0 = db * 32 + 8 * gi + 4 * h;
          uint2 st;
          st.x = pack_bf16x2(acc_o[qb][db][4 * gi + 0] * inv, acc_o[qb][db][4 * gi + 1] * inv);
          st.y = pack_bf16x2(acc_o[qb][db][4 * gi + 2] * inv, acc_o[qb][db][4 * gi + 3] * inv);
          *reinterpret_cast<uint2 *>(orow + d0) = st;
        }
    }
    return;
  }

  // split-KV: write this split's partial result
  const int64_t split_stride = static_cast<int64_t>(p.total_q) * p.num_q_heads;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    if (!valid[qb]) continue;
    const int64_t rowidx = qoff[qb] / D;     // (cu + i) * Hq + hq
    float *po = p.part_o + (split * split_stride + rowidx) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        const int d0 = db * 32 + 8 * gi + 4 * h;
        *reinterpret_cast<float4 *>(po + d0) =
            make_float4(acc_o[qb][db][4 * gi + 0], acc_o[qb][db][4 * gi + 1],
                        acc_o[qb][db][4 * gi + 2], acc_o[qb][db][4 * gi + 3]);
      }
    if (h == 0) {
      float *pml = p.part_ml + (split * split_stride + rowidx) * 2;
      *reinterpret_cast<float2 *>(pml) = make_float2(m_run[qb], l_tot[qb]);
    }
  }
  __threadfence();
  __syncthreads();
  const int64_t group = (static_cast<int64_t>(bg)) * p.qtiles + qtile;
  if (tid == 0) sh_last = atomicAdd(&p.counters[group], 1u);
  __syncthreads();
  if (sh_last != static_cast<uint32_t>(nsplit - 1)) return;
  __threadfence();

  // last split of this query tile: merge all splits in split order
  const int rows_here = min(kRowsPerTile, M - row0);
  constexpr int D4 = D / 4;
  for (int item = tid; item < rows_here * D4; item += kT) {
    const int rr = row0 + item / D4;
    const int d0 = (item % D4) * 4;
    const int i = rr / G;
    if (cu + i >= p.total_q) continue;
    const int hq = g * G + rr % G;
    const int64_t rowidx = static_cast<int64_t>(cu + i) * p.num_q_heads + hq;
    float mmax = kNegInf;
    for (int sp = 0; sp < nsplit; ++sp) mmax = fmaxf(mmax, p.part_ml[(sp * split_stride + rowidx) * 2]);
    float lsum = 0.f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sp = 0; sp < nsplit; ++sp) {
      const float2 ml = *reinterpret_cast<const float2 *>(p.part_ml + (sp * split_stride + rowidx) * 2);
      if (ml.x == kNegInf) continue;          // split saw no key of this row
      const float wgt = __builtin_amdgcn_exp2f(ml.x - mmax);
      lsum += wgt * ml.y;
      const float4 po = *reinterpret_cast<const float4 *>(p.part_o + (sp * split_stride + rowidx) * D + d0);
      o.x += wgt * po.x;
      o.y += wgt * po.y;
      o.z += wgt * po.z;
      o.w += wgt * po.w;
    }
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    uint2 st;
    st.x = pack_bf16x2(o.x * inv, o.y * inv);
    st.y = pack_bf16x2(o.z * inv, o.w * inv);
    *reinterpret_cast<uint2 *>(p.out + rowidx * D + d0) = st;
  }
  if (tid == 0) p.counters[group] = 0u;    // ready for the next call
}

template <int D, int MODE>
hipError_t launch_t(const AttnParams &p, hipStream_t stream) {
  const int64_t grid = p.units_per_xcd * kXcds;
  hipLaunchKernelGGL((window_attention_kernel<D, MODE>), dim3(static_cast<unsigned>(grid)), dim3(kT), 0,
                     stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_window_attention(const AttnParams &p, int head_dim, int mask_mode, hipStream_t stream) {
  if (head_dim == 128) return mask_mode == 1 ? launch_t<128, 1>(p, stream) : launch_t<128, 0>(p, stream);
  return mask_mode == 1 ? launch_t<64, 1>(p, stream) : launch_t<64, 0>(p, stream);
}

}  // namespace mbe
