// Confidence-based edit selection over vocabulary logits, gfx950.
//
// Paper, Sec. "Configurable threshold decoding", Eq. (1): per position, the
// prediction is the highest-probability token and its confidence is that
// probability; a visible token is overwritten (the token-to-token set) when
// the prediction differs from it and the confidence clears the threshold.
// MBE keeps this rule for its cross-block passes (Sec. "Training-Free MBE
// Decoding").  Ties go to the lowest index; the test is conf >= threshold.
//
// One HBM pass per row.  Each workgroup (256 threads) reduces one chunk of a
// row; each thread streams 16-byte bf16 vectors (the next iteration's two
// loads in flight while the current one is reduced) and keeps
//   m       its running maximum,
//   s       sum of 2^(x log2(e) - mc), mc = m log2(e) rounded to fp32,
//           rescaled when m grows,
//   it_max  the iteration where m was first reached.
// The exponent is one FMA per element.  Every exponent is off by the same
// delta = m log2(e) - mc (the rounding residual of mc), so the confidence of
// the maximum is 2^delta / s, and the entropy, which does not depend on the
// reference, needs no correction.
// Elements of one thread are visited in increasing index order, so its first
// occurrence of m lies in iteration it_max.  Threads merge (max, rescaled
// sum) in a fixed tree; then only the threads whose own maximum equals the
// chunk maximum re-read their iteration it_max to find its first index, and a
// min over the workgroup picks the lowest.  This keeps the argmax bookkeeping
// out of the per-element loop at the cost of a few cache lines per chunk.
// Rows split over several workgroups (few rows) write partials that a small
// finalize kernel merges in chunk order, so results are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "internal.h"

namespace mbe {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kU = kEsVecPerThread;
constexpr int kT = kEsThreads;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_at(const uint16_t *p) {
  return __uint_as_float(static_cast<uint32_t>(*p) << 16);
}

// Exponent arguments below this are exactly 0 after exp2 in fp32.  The
// entropy sum adds 2^y * y; a -inf logit would add 0 * (-inf).  The main pass
// does not clamp; a NaN sum sends the chunk through a second pass that clamps
// y here (only rows holding -inf logits take it).
constexpr float kYMin = -256.f;

// The reference of a running maximum m: m log2(e) rounded to fp32.  All sums
// are kept relative to it.  The product is formed by its own instruction:
// fused into a following subtraction (d = ref(m) - ref(M)) it would lose the
// rounding that the sums were accumulated against.
__device__ __forceinline__ float ref_of(float m) {
  float r;
  asm("v_mul_f32 %0, %1, %2" : "=v"(r) : "v"(m), "v"(kLog2e));
  return r;
}

// Merge partial (m, s, t) with (m2, s2, t2): the sums are rescaled to the
// common max M.  With d = ref(m) - ref(M): s -> 2^d s, t -> 2^d (t + d s).
template <bool ENT>
__device__ __forceinline__ void merge_ms(float &m, float &s, float &t, float m2, float s2, float t2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;     // both empty so far
  float a = 0.f, b = 0.f, ta = 0.f, tb = 0.f;
  const float rM = ref_of(M);
  if (m != -INFINITY) {
    const float d = ref_of(m) - rM;
    const float f = __builtin_amdgcn_exp2f(d);
    a = s * f;
    if (ENT) ta = f * __builtin_fmaf(d, s, t);
  }
  if (m2 != -INFINITY) {
    const float d = ref_of(m2) - rM;
    const float f = __builtin_amdgcn_exp2f(d);
    b = s2 * f;
    if (ENT) tb = f * __builtin_fmaf(d, s2, t2);
  }
  s = a + b;
  if (ENT) t = ta + tb;
  m = M;
}

// Merge partial (m, s, t, i) with (m2, s2, t2, i2): larger max wins, equal
// maxima keep the lower index.
template <bool ENT>
__device__ __forceinline__ void merge(float &m, float &s, float &t, int32_t &i, float m2, float s2, float t2,
                                      int32_t i2) {
  i = (m > m2) ? i : ((m2 > m) ? i2 : min(i, i2));
  merge_ms<ENT>(m, s, t, m2, s2, t2);
}

// Entropy in nats from s = sum 2^y and t = sum 2^y y:
// H = -sum p ln p with p = 2^y / s, i.e. ln 2 (log2 s - t / s).
__device__ __forceinline__ float entropy_nats(float s, float t) {
  return 0.69314718055994531f * (log2f(s) - t / s);
}

// max(a, b, c) in one instruction.  fmaxf would first quiet every input
// (one more instruction each): the compiler cannot tell that floats made
// from bf16 bits by shifts are not signalling NaNs.  NaN logits are outside
// the contract; -inf is handled like any value.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Maximum of the 8 kU logits of one iteration, three at a time (a tree of
// about 4 kU three-input maxima).
__device__ __forceinline__ float max_iter(const float (&x)[kU][8]) {
  constexpr int N = 8 * kU;
  float v[N];
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = x[i / 8][i % 8];
  int n = N;
#pragma unroll
  for (int level = 0; level < 8; ++level) {
    if (n == 1) break;
    int m = 0;
#pragma unroll
    for (int i = 0; i < N; i += 3) {
      if (i >= n) break;
      if (i + 2 < n) v[m] = max3(v[i], v[i + 1], v[i + 2]);
      else if (i + 1 < n) v[m] = max3(v[i], v[i + 1], v[i + 1]);
      else v[m] = v[i];
      ++m;
    }
    n = m;
  }
  return v[0];
}

// Eight bf16 logits of one 16-byte vector as floats.
__device__ __forceinline__ void unpack8(const u32x4 &w, float x[8]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    x[2 * k] = bf16_lo(w[k]);
    x[2 * k + 1] = bf16_hi(w[k]);
  }
}

// Streaming load of one 16-byte vector: each logit is read once, so it is
// not kept in cache.
__device__ __forceinline__ u32x4 load16(const uint16_t *row, int64_t unit) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(row + unit * 8));
}

// Loads vector unit `unit` (elements 8*unit .. 8*unit+7) as 8 floats; elements
// at or beyond `end` read as -inf.
template <bool VEC>
__device__ __forceinline__ void load_unit(const uint16_t *row, int64_t unit, int64_t end, float x[8]) {
  const int64_t e0 = unit * 8;
  if (VEC && e0 + 8 <= end) {
    unpack8(load16(row, unit), x);
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = (e0 + k < end) ? bf16_at(row + e0 + k) : -INFINITY;
  }
}

// The token-to-token decision for one row from its (max, argmax, sum), or,
// for the threshold update, the row's prediction, confidence and entropy.
template <bool ENT>
__device__ __forceinline__ void decide(const EsParams &p, int64_t row, float m, float s, float t, int32_t idx) {
  // the maximum's own term is 2^delta, delta = m log2(e) - ref(m) exactly
  // (0 when the product is exact, e.g. on a constant row of small integers)
  const float delta = __builtin_fmaf(m, kLog2e, -ref_of(m));
  const float conf = (delta == 0.f ? 1.0f : __builtin_amdgcn_exp2f(delta)) / s;   // correctly rounded division
  if (p.update) {
    p.pred[row] = idx;
    p.conf[row] = (m == -INFINITY) ? __builtin_nanf("") : conf;
    if (ENT) p.entropy[row] = entropy_nats(s, t);
    return;
  }
  const int32_t cur = p.cur[row];
  const bool change = (m != -INFINITY) && (idx != cur) && (conf >= p.threshold);
  p.conf[row] = (m == -INFINITY) ? __builtin_nanf("") : conf;
  p.new_tokens[row] = change ? idx : cur;
  p.changed[row] = change ? 1 : 0;
}

template <bool VEC, bool ENT>
__global__ __launch_bounds__(kT) void edit_select_kernel(EsParams p) {
  __shared__ float sh_m[kT / 64];
  __shared__ float sh_s[kT / 64];
  __shared__ float sh_t[kT / 64];
  __shared__ int32_t sh_i[kT / 64];
  if (p.changed_count && blockIdx.x == 0 && threadIdx.x == 0) *p.changed_count = 0;   // counted per block later
  if (p.gate && *p.gate == 0) return;     // gated off: the block step keeps every row

  const int64_t wg = blockIdx.x;
  const int64_t row = wg / p.chunks;
  const int32_t chunk = static_cast<int32_t>(wg % p.chunks);
  const int tid = threadIdx.x;
  const uint16_t *rowp = p.logits + row * p.ld;
  const int64_t c0 = static_cast<int64_t>(chunk) * p.chunk_len;
  const int64_t c1 = min(p.vocab, c0 + p.chunk_len);
  const int64_t u0 = c0 / 8;
  const int64_t u1 = (c1 + 7) / 8;

  float m = -INFINITY, s = 0.f, t = 0.f;
  int32_t it_max = -1;
  int32_t it = 0;
  // One iteration's 16 logits of this thread into the running (m, s, t).
  auto accumulate = [&](const float (&x)[kU][8], auto clamp) {
    const float cm = max_iter(x);
    if (cm > m) {
      if (m == -INFINITY) {
        s = 0.f;
        t = 0.f;
      } else {
        const float d = ref_of(m) - ref_of(cm);
        const float f = __builtin_amdgcn_exp2f(d);
        if (ENT) t = f * __builtin_fmaf(d, s, t);
        s *= f;
      }
      m = cm;
      it_max = it;
    }
    const float nref = (m == -INFINITY) ? 0.f : -ref_of(m);
    float acc = 0.f, acct = 0.f;
#pragma unroll
    for (int j = 0; j < kU; ++j)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        float y = __builtin_fmaf(x[j][k], kLog2e, nref);
        if constexpr (decltype(clamp)::value) y = fmaxf(y, kYMin);
        const float e = __builtin_amdgcn_exp2f(y);
        acc += e;
        if (ENT) acct = __builtin_fmaf(e, y, acct);
      }
    s += acc;
    if (ENT) t += acct;
  };
  // The whole chunk: iterations whose units all lie inside the chunk with
  // unguarded vector loads, the next iteration's loads issued before the
  // current one is reduced; then at most one guarded iteration.
  auto pass = [&](auto clamp) {
    m = -INFINITY;
    s = 0.f;
    t = 0.f;
    it_max = -1;
    it = 0;
    constexpr int64_t per_iter = kT * kU;
    int64_t base = u0;
    if constexpr (VEC) {
      const int64_t u_full = c1 / 8;      // units [u0, u_full) hold 8 logits of the chunk each
      const int64_t n_full = u_full > u0 ? (u_full - u0) / per_iter : 0;
      if (n_full > 0) {
        u32x4 w[kU];
#pragma unroll
        for (int j = 0; j < kU; ++j) w[j] = load16(rowp, base + j * kT + tid);
        for (int64_t i = 0; i < n_full; ++i, base += per_iter, ++it) {
          float x[kU][8];
#pragma unroll
          for (int j = 0; j < kU; ++j) unpack8(w[j], x[j]);
          if (i + 1 < n_full) {
#pragma unroll
            for (int j = 0; j < kU; ++j) w[j] = load16(rowp, base + per_iter + j * kT + tid);
          }
          accumulate(x, clamp);
        }
      }
    }
    for (; base < u1; base += per_iter, ++it) {
      float x[kU][8];
#pragma unroll
      for (int j = 0; j < kU; ++j) {
        const int64_t unit = base + j * kT + tid;
        if (unit < u1) {
          load_unit<VEC>(rowp, unit, c1, x[j]);
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) x[j][k] = -INFINITY;
        }
      }
      accumulate(x, clamp);
    }
  };
  pass(std::false_type{});

  // (max, rescaled sum) over the workgroup: wave butterfly, then the four
  // wave results in wave order.  Afterwards every thread holds the same
  // (m, s, t).
  const int wave = tid / 64;
  float m_own = m;
  auto reduce = [&]() {
    m_own = m;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float m2 = __shfl_xor(m, o);
      const float s2 = __shfl_xor(s, o);
      const float t2 = ENT ? __shfl_xor(t, o) : 0.f;
      merge_ms<ENT>(m, s, t, m2, s2, t2);
    }
    if ((tid & 63) == 0) {
      sh_m[wave] = m;
      sh_s[wave] = s;
      sh_t[wave] = t;
    }
    __syncthreads();
    m = sh_m[0];
    s = sh_s[0];
    t = sh_t[0];
#pragma unroll
    for (int w = 1; w < kT / 64; ++w) merge_ms<ENT>(m, s, t, sh_m[w], sh_s[w], sh_t[w]);
  };
  reduce();
  if constexpr (ENT) {
    if (t != t) {          // the chunk holds a -inf logit: clamped second pass
      __syncthreads();     // every thread has read the shared partials
      pass(std::true_type{});
      reduce();
    }
  }

  // First index of the chunk maximum.  Only threads whose own maximum equals
  // it look: their first occurrence lies in iteration it_max, re-read once
  // (the other threads read nothing more, so the re-read costs a few cache
  // lines per chunk instead of one per thread).
  int32_t idx = INT32_MAX;
  if (m != -INFINITY && m_own == m) {
    const int64_t base = u0 + static_cast<int64_t>(it_max) * kT * kU;
    for (int j = 0; j < kU && idx == INT32_MAX; ++j) {
      const int64_t unit = base + j * kT + tid;
      if (unit >= u1) break;
      float x[8];
      load_unit<VEC>(rowp, unit, c1, x);
      for (int k = 0; k < 8; ++k) {
        if (x[k] == m) {
          idx = static_cast<int32_t>(unit * 8 + k);
          break;
        }
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) idx = min(idx, __shfl_xor(idx, o));
  if ((tid & 63) == 0) sh_i[wave] = idx;
  __syncthreads();
  if (tid != 0) return;
#pragma unroll
  for (int w = 0; w < kT / 64; ++w) idx = min(idx, sh_i[w]);

  if (p.chunks > 1) {     // merged by the finalize kernel
    p.partials[row * p.chunks + chunk] = EsPartial{m, s, idx, t};
    return;
  }
  decide<ENT>(p, row, m, s, t, idx);
}

// Rows reduced in several chunks: one wave per row merges the chunk partials
// (the kernel boundary makes them visible).  Lane l merges chunks l, l + 64,
// ... in order, then a butterfly combines the lanes; every step is a fixed,
// commutative merge, so the result is the same on every lane and in every run.
template <bool ENT>
__global__ __launch_bounds__(256) void edit_select_finalize_kernel(EsParams p) {
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= p.rows || (p.gate && *p.gate == 0)) return;
  const int lane = threadIdx.x & 63;
  const EsPartial *pp = p.partials + row * p.chunks;
  float m = -INFINITY, s = 0.f, t = 0.f;
  int32_t idx = INT32_MAX;
  for (int c = lane; c < p.chunks; c += 64) {
    const EsPartial q = pp[c];
    merge<ENT>(m, s, t, idx, q.m, q.s, q.t, q.idx);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float m2 = __shfl_xor(m, o);
    const float s2 = __shfl_xor(s, o);
    const float t2 = ENT ? __shfl_xor(t, o) : 0.f;
    const int32_t i2 = __shfl_xor(idx, o);
    merge<ENT>(m, s, t, idx, m2, s2, t2, i2);
  }
  if (lane == 0) decide<ENT>(p, row, m, s, t, idx);
}

// Threshold update, second step: one workgroup per block of block_size rows
// applies the mask-to-token set, the force-unmask and the token-to-token set
// to the rows' predictions and confidences.  Each row's current token is read
// and its new token written by the same thread, so new_tokens may be
// cur_tokens itself (an in-place update).
__global__ __launch_bounds__(256) void threshold_block_kernel(EsParams p) {
  __shared__ unsigned long long sh_best;
  __shared__ int32_t sh_changed;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * p.block_size;
  const int tid = threadIdx.x;
  if (p.gate && *p.gate == 0) {
    // gated off: the pass changes nothing (its rows were not reduced)
    for (int i = tid; i < p.block_size; i += 256) {
      p.action[r0 + i] = 0;
      p.new_tokens[r0 + i] = p.cur[r0 + i];
    }
    if (tid == 0) p.block_changed[blockIdx.x] = 0;
    return;
  }
  if (tid == 0) {
    sh_best = 0;
    sh_changed = 0;
  }
  __syncthreads();
  bool any_gamma = false, any_masked = false;
  for (int i = tid; i < p.block_size; i += 256) {
    const int64_t r = r0 + i;
    const bool masked = p.cur[r] == p.mask_id;
    const float c = p.conf[r];
    any_masked |= masked;
    any_gamma |= masked && c > p.omega_mask;
    if (masked) {
      // highest confidence first, then the lowest row: conf is positive, so its
      // bits order like the value
      const unsigned long long key = (static_cast<unsigned long long>(__float_as_uint(c)) << 32) |
                                     (0xffffffffu - static_cast<uint32_t>(i));
      atomicMax(&sh_best, key);
    }
  }
  any_gamma = __syncthreads_or(any_gamma);
  any_masked = __syncthreads_or(any_masked);
  const int forced = (any_masked && !any_gamma) ? static_cast<int>(0xffffffffu - static_cast<uint32_t>(sh_best)) : -1;
  int changed = 0;
  for (int i = tid; i < p.block_size; i += 256) {
    const int64_t r = r0 + i;
    const int32_t cur = p.cur[r];
    const int32_t a = p.pred[r];
    const float c = p.conf[r];
    uint8_t act = 0;
    if (cur == p.mask_id) {
      if (c > p.omega_mask) act = 1;
      else if (i == forced) act = 2;
    } else if (a != cur && c >= p.threshold) {
      act = 3;
    }
    p.action[r] = act;
    p.new_tokens[r] = act ? a : cur;
    changed += act != 0;
  }
  if (changed) atomicAdd(&sh_changed, changed);
  __syncthreads();
  if (tid == 0) {
    p.block_changed[blockIdx.x] = sh_changed != 0;
    if (p.changed_count && sh_changed) atomicAdd(p.changed_count, sh_changed);
  }
}

}  // namespace

template <bool ENT>
hipError_t launch_rows(const EsParams &p, bool vector_loads, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(p.rows * p.chunks));
  if (vector_loads)
    hipLaunchKernelGGL((edit_select_kernel<true, ENT>), grid, dim3(kT), 0, stream, p);
  else
    hipLaunchKernelGGL((edit_select_kernel<false, ENT>), grid, dim3(kT), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.chunks == 1) return e;
  hipLaunchKernelGGL(edit_select_finalize_kernel<ENT>, dim3(static_cast<unsigned>((p.rows + 3) / 4)), dim3(256), 0,
                     stream, p);
  return hipGetLastError();
}

hipError_t launch_edit_select(const EsParams &p, bool vector_loads, hipStream_t stream) {
  return launch_rows<false>(p, vector_loads, stream);
}

hipError_t launch_threshold_update(const EsParams &p, bool vector_loads, hipStream_t stream) {
  hipError_t e = p.entropy ? launch_rows<true>(p, vector_loads, stream) : launch_rows<false>(p, vector_loads, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(threshold_block_kernel, dim3(static_cast<unsigned>(p.rows / p.block_size)), dim3(256), 0, stream,
                     p);
  return hipGetLastError();
}

}  // namespace mbe
