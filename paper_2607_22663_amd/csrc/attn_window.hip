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
//   position i of query head g*G + hl.  A workgroup owns 256 such rows and
//   one split of the key range; its 8 waves (two per
//   SIMD, so that one wave's LDS reads and waits overlap the other's work)
//   own 32 rows each, one 32-row MFMA column block.
//
// Contractions on bf16 MFMA (v_mfma_f32_32x32x16_bf16)
//   S^T = K . Q^T : A = 32 keys x 16 dims from LDS, B = Q^T from registers.
//                  The result holds one query per lane (column), so softmax
//                  statistics stay in the lane; only the two 32-lane halves,
//                  which hold different keys of the same query, exchange.
//   O^T += V^T . P^T : A = 32 dims x 16 keys of V^T from LDS, B = P^T taken
//                  straight from the S^T accumulators.  Keys are assigned to
//                  MFMA rows through a fixed permutation (swap of bits 2 and 3
//                  of the row index) so that the 8 keys a lane contributes to
//                  one P.V step are 8 consecutive keys: with token-minor V
//                  pages ([D][16]) that is one 16-byte LDS read per operand;
//                  with token-major V pages ([16][D], like K) two transposing
//                  LDS reads (ds_read_b64_tr_b16), each giving a lane 4 keys
//                  of its dim.
//
// Softmax: base 2, fp32, against a fixed reference per row instead of a
// running maximum, so inside the key loop the O accumulators are touched by
// MFMA only.  The reference is the row's maximum over the first 32 keys of
// its split.
// Later exponentials 2^(s - ref) may exceed 1; bf16 P and fp32 sums share
// fp32's exponent range, so nothing overflows unless a later score exceeds
// the reference by about 2^127.  The row sum is checked once at the end of
// the key range: if any sum exceeds 2^64 (or is not finite) the workgroup
// makes a max-only run over its keys and then a full run with the true
// maximum as reference, where no exponential exceeds 1.
//
// Split-KV: when the work would not fill the chip, long key ranges are cut
// into kv_chunk-key splits.  Each split writes unnormalised O, its reference
// and its sum; a second, small kernel merges them in split order.
//
// K/V tiles of 64 keys (four 16-token pages gathered through the page table)
// go from HBM straight into LDS (global_load_lds_dwordx4, no registers), four
// buffers with three tiles in flight.  Long units with token-minor V run a
// software-pipelined key loop instead (PIPE): the scores of the next 32-key
// block are formed on the matrix cores while the current block is
// exponentiated, over five buffers.  Waves w and w + 4 fetch page w % 4 of
// each tile, half of it each: each load instruction reads 1 KB of one page
// (a scalar page base plus a fixed lane offset) and fills 1 KB of LDS.  K rows land XOR-swizzled, a
// token-minor V page ([D][16 keys]) with the two 8-key halves of every other
// group of 8 dims swapped, a token-major one row by row with its own swizzle,
// so that the MFMA operand reads are free of bank conflicts.  Work groups
// (split, sequence, KV head) are dealt round-robin to the XCDs, and the query
// tiles sharing a key range run back to back on the same XCD (shared L2).
//
// Targeted refresh and early exit (Sec. "Infrastructure Optimization", cache
// control; the pass loop of Sec. "Training-Free MBE Decoding"): with block
// flags only the rows of flagged window blocks are computed and written, and
// with a device gate the whole call does nothing when the gate reads 0.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "internal.h"

namespace mbe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kT = kWaves * 64;
constexpr int QB = kRowsPerWave / 32;   // 32-row query blocks (MFMA columns) per wave
constexpr int kPageWaves = kWaves / 4;  // waves that share the direct loads of one page
constexpr float kNegInf = -INFINITY;
constexpr float kSumLimit = 0x1p64f;   // row sums above this trigger the exact rerun
constexpr bf16x2 kOnes2 = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};

template <int D>
struct Tile {
  static constexpr int kRowChunks = D / 8;                   // 16-byte chunks per K row
  static constexpr int kPageBytes = kPageSize * D * 2;       // one page of one KV head, K or V
  static constexpr int kKBytes = kKeyTile * D * 2;           // K: 64 keys x D, row-major, swizzled
  static constexpr int kVBytes = D * kKeyTile * 2;           // V: 4 pages of [D][16 keys]
  static constexpr int kBufBytes = kKBytes + kVBytes;
  static constexpr int kLoads = kPageBytes / 1024;           // 1 KB direct loads per page, K and V each
  static constexpr int kWaveLoads = kLoads / kPageWaves;     // of those, per wave
  static_assert(kLoads * 4 * 1024 == kKBytes, "four pages per tile");
  static_assert(kWaveLoads * kPageWaves == kLoads, "the waves of a page share its loads evenly");
};

// LDS chunk position of global chunk j of K row r (XOR swizzle; an involution).
template <int D>
__device__ __forceinline__ int k_swz(int r) {
  return D == 128 ? (r & 15) : ((r >> 1) & 7);
}
// LDS chunk position of global chunk j of a token-major V row r: j ^ v_swz(r).
// A transposing read of a half-wave covers 4 consecutive key rows and 32
// dims (4 chunks); rows r..r+3 land on disjoint 16-byte banks groups.
template <int D>
__device__ __forceinline__ int v_swz(int r) {
  return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1);
}
// LDS half (16 bytes: keys 0-7 or 8-15 of a page) of half q of V dim row d.
// The 16 lanes that LDS serves together read dims c .. c+15 of one half;
// without the swap dims c and c+8 would share banks.
__device__ __forceinline__ int v_half(int d, int q) { return q ^ ((d >> 3) & 1); }
// Bit swap 2<->3 of a row index in 0..31: MFMA row -> key within a 32-key block.
__device__ __forceinline__ int perm_row(int r) {
  return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Two floats to two bf16, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = __builtin_convertvector(f32x2{lo, hi}, bf16x2);
  return __builtin_bit_cast(uint32_t, v);
}

// s_waitcnt immediate that waits for vector-memory count <= n only
// (vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt fields at their maxima).
constexpr int wait_vmcnt(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xF00; }

// Workgroup barrier for LDS only, without the memory fence of
// __syncthreads(): that fence would also wait for every direct HBM->LDS load
// still in flight.  The caller first waits for the loads it needs; pending
// LDS writes of this wave are waited for here.  The memory clobber keeps the
// compiler from moving LDS accesses across the barrier.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ bf16x8 lds_read8(const char *base, int byte_off) {
  return *reinterpret_cast<const bf16x8 *>(base + byte_off);
}

// Transposing LDS read (ds_read_b64_tr_b16): within each group of 16 lanes,
// lane i receives element i % 4 of the 8-byte pieces that lanes i / 4,
// i / 4 + 4, i / 4 + 8 and i / 4 + 12 address.
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x4 lds_read_tr4(const char *at) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4 *)(at));
  return __builtin_bit_cast(bf16x4, v);
}

typedef const __attribute__((address_space(4))) int32_t const_i32;

// A load that stays where it is written: the compiler would otherwise move a
// plain load into the branch that uses it, behind an earlier branch's wait,
// so that loads meant to be in flight together are issued one after another.
// (A relaxed atomic load is never moved; at workgroup scope it is an ordinary
// vector load.)
__device__ __forceinline__ int32_t load_now(const int32_t *ptr) {
  return __hip_atomic_load(ptr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Page id of page `wv` (0..3) of the 64-key tile starting at key0, read with a scalar
// load (the page table is constant during the kernel), or with load_now when
// kNow (the first tile's, read together with the lengths).  Slots past the
// table row are clamped into it and ids into the pool; such pages only feed
// keys that are masked and whose V rows are zeroed.
template <bool kNow = false>
__device__ __forceinline__ int wave_page(const AttnParams &p, int b, int key0, int wv,
                                         std::integral_constant<bool, kNow> = {}) {
  const int64_t row = static_cast<int64_t>(b) * p.max_pages;
  const int slot = min(key0 / kPageSize + wv, p.max_pages - 1);
  int pid;
  if constexpr (kNow) pid = __builtin_amdgcn_readfirstlane(load_now(p.page_table + row + slot));
  else pid = ((const_i32 *)(p.page_table))[row + slot];
  return min(max(pid, 0), p.num_pages - 1);
}

// Per-lane byte offsets, within one K page, of the chunks that the direct
// loads j = 0 .. kWaveLoads-1 of part `part` of a page fetch (part p takes
// the page's loads p * kWaveLoads ..): page load i fills LDS slots
// 64 i + lane of the page, slot s holding chunk (s % RC) ^ k_swz(row) of key
// row s / RC.  They do not depend on the tile.
template <int D>
__device__ __forceinline__ void k_load_offsets(uint32_t (&koff)[Tile<D>::kWaveLoads], int part) {
  constexpr int RC = Tile<D>::kRowChunks;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < Tile<D>::kWaveLoads; ++j) {
    const int row = ((part * Tile<D>::kWaveLoads + j) * 64 + lane) / RC;   // key within the page
    const int chunk = (lane % RC) ^ k_swz<D>(row);
    koff[j] = static_cast<uint32_t>(row * (2 * D) + chunk * 16);
  }
}

// The same for a token-major V page: v_swz depends only on the row's low bits
// (2 for D = 128, 3 for D = 64), which a lane keeps in every load, so page
// load i reads lane offset + i KB.
template <int D>
__device__ __forceinline__ uint32_t vt_load_offset() {
  constexpr int RC = Tile<D>::kRowChunks;
  const int lane = threadIdx.x & 63;
  const int row = lane / RC;
  return static_cast<uint32_t>(row * (2 * D) + (((lane % RC) ^ v_swz<D>(row)) << 4));
}

// Cache policy of the K/V loads: nontemporal (the `nt` bit).  A tile is read
// by the workgroups of one (sequence, KV head, split) at about the same time
// and not again in the call, so its lines are marked for early eviction
// rather than kept in the L2 and infinity cache; on the HBM-bound shapes
// (one or two window blocks) this is 3-5% faster, elsewhere the same.
constexpr int kStreamLoad = 2;

// Issues this wave's direct HBM->LDS loads of one 64-key tile into `buf`:
// waves w and w + 4 fetch page w % 4 of the tile, each one part (half) of its
// K rows (swizzled) and of its V page ([D][16 keys], 8-key halves placed by
// v_half; token-major: rows like K).  Each load reads 1 KB from one page, so
// its address is a scalar page base plus a loop-invariant lane offset,
// koff[j] for K and voff for V (the empty asm statements keep the two apart,
// which selects the scalar-base form of the load instead of 64-bit vector
// address arithmetic).
template <int D, int VT>
__device__ __forceinline__ void load_tile(const AttnParams &p, int g, int wpage, int part, int pid,
                                          uint32_t *koff, uint32_t &voff, char *buf) {
  constexpr int PB = Tile<D>::kPageBytes;
  pid = __builtin_amdgcn_readfirstlane(pid);   // wave-uniform; lets it live in a scalar register
  const int64_t page = (static_cast<int64_t>(pid) * p.num_kv_heads + g) * PB;
  uint64_t kbase = reinterpret_cast<uint64_t>(p.k_pages) + page;
  uint64_t vbase = reinterpret_cast<uint64_t>(p.v_pages) + page;
  asm("" : "+s"(kbase), "+s"(vbase));
  constexpr int WL = Tile<D>::kWaveLoads;
  char *kdst = buf + wpage * PB + part * WL * 1024;
  char *vdst = buf + Tile<D>::kKBytes + wpage * PB + part * WL * 1024;
#pragma unroll
  for (int j = 0; j < WL; ++j) {
    asm("" : "+v"(koff[j]) : "s"(pid));
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(kbase) + koff[j], (lds_void *)(kdst + j * 1024),
                                     16, 0, kStreamLoad);
  }
  // token-minor V: LDS slot i*64 + lane of the page is dim (32i + lane/2),
  // half lane&1, and holds that dim's half v_half(d, lane & 1) (the swap is
  // its own inverse).  Token-major V: rows like K, swizzled by v_swz.
  asm("" : "+v"(voff) : "s"(pid));
#pragma unroll
  for (int j = 0; j < WL; ++j)
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(vbase + (part * WL + j) * 1024) + voff,
                                     (lds_void *)(vdst + j * 1024), 16, 0, kStreamLoad);
}

// Zeroes V entries of keys at or past `nvalid` (tile-relative) so that
// unread page tails (which may hold anything) cannot reach the P.V product.
template <int D, int VT>
__device__ __forceinline__ void zero_v_tail(char *buf, int nvalid) {
  if constexpr (VT) {     // token-major: whole key rows [nvalid, 64) of the tile
    uint4 *vs = reinterpret_cast<uint4 *>(buf + Tile<D>::kKBytes);
    constexpr int RC = Tile<D>::kRowChunks;
    for (int i = nvalid * RC + static_cast<int>(threadIdx.x); i < kKeyTile * RC; i += kT) vs[i] = make_uint4(0, 0, 0, 0);
    return;
  }
  uint16_t *vs = reinterpret_cast<uint16_t *>(buf + Tile<D>::kKBytes);
  for (int s = threadIdx.x; s < 4 * D; s += kT) {   // row s: page s / D, dim s % D, 16 keys
    const int k0 = (s / D) * kPageSize;
    if (k0 + kPageSize <= nvalid) continue;
    uint16_t *e = vs + s * kPageSize;
    const int d = s % D;
#pragma unroll
    for (int k = 0; k < kPageSize; ++k)
      if (k0 + k >= nvalid) e[v_half(d, k >> 3) * 8 + (k & 7)] = 0;
  }
}

// KS = 1: the eight waves own 32 rows each.  KS = 2 (at most 128 rows per
// sequence and KV head): waves w and w + 4 own the same 32 rows and split the
// keys, wave w taking the first and wave w + 4 the second 32-key block of
// every tile; their partial results are added at the end.
// Phase timeline (profiling builds only, compiled with -DMBE_TIMELINE): thread
// 0 of each of the first kTimelineWgs workgroups records the 100 MHz real-time
// counter at entry (0), once its lengths are read (1), when its first tile is
// in LDS (2), after its key loop (3) and once its stores have completed (4),
// and the shader-clock counter at entry (6) and end (7).  A workgroup that
// exits early leaves its later entries as they were.  Product builds record
// nothing.
#ifdef MBE_TIMELINE
constexpr int kTimelineWgs = 8192;
__device__ unsigned long long g_timeline[kTimelineWgs * 8];
#define MBE_TL(k, clock)                                                                     \
  do {                                                                                       \
    if (threadIdx.x == 0 && blockIdx.x < kTimelineWgs)                                       \
      g_timeline[blockIdx.x * 8 + (k)] = clock;                                              \
  } while (0)
#define MBE_TL_REAL(k) MBE_TL(k, __builtin_amdgcn_s_memrealtime())
#define MBE_TL_CYCLES(k) MBE_TL(k, __builtin_amdgcn_s_memtime())
#define MBE_TL_END()                                                                         \
  do {                                                                                       \
    __builtin_amdgcn_s_waitcnt(0);                                                           \
    MBE_TL_REAL(4);                                                                          \
    MBE_TL_CYCLES(7);                                                                        \
  } while (0)
#else
#define MBE_TL_REAL(k) do {} while (0)
#define MBE_TL_CYCLES(k) do {} while (0)
#define MBE_TL_END() do {} while (0)
#endif

template <int D, int MODE, int KS, int VT, int PIPE>
__global__ __launch_bounds__(kT, 1) void window_attention_kernel(AttnParams p) {
  static_assert(!PIPE || (KS == 1 && QB == 1), "the pipelined loop holds one 32-row block per wave");
  MBE_TL_REAL(0);
  MBE_TL_CYCLES(6);
  // K/V tile buffers (separate objects, so the compiler can tell which
  // in-flight direct loads a read depends on): four with three tiles in
  // flight, or five in the pipelined loop (PIPE)
  __shared__ __align__(1024) char lds0[Tile<D>::kBufBytes];
  __shared__ __align__(1024) char lds1[Tile<D>::kBufBytes];
  __shared__ __align__(1024) char lds2[Tile<D>::kBufBytes];
  __shared__ __align__(1024) char lds3[Tile<D>::kBufBytes];
  __shared__ __align__(1024) char lds4[PIPE ? Tile<D>::kBufBytes : 1024];   // the pipelined loop's fifth

  // ---- work unit.  Workgroup id % 8 is the XCD that runs it.  With a
  // dispatch table the host has placed every unit (groups dealt largest
  // first to the least-loaded XCD, each XCD's longest units first).
  // Otherwise groups (split, sequence rank, KV head), split slowest, are dealt
  // to the XCDs round-robin, so that every XCD gets the same mix of first and
  // later splits (later splits of short sequences have no work).  Either way
  // the qtiles query tiles of a group, which read the same keys, take
  // consecutive slots of one XCD so that the second finds the keys in its L2.
  // gated off: the call does nothing (the gate is read together with the
  // work unit and checked once both are in)
  const int32_t gate = load_now(p.gate ? p.gate : p.prefix_lens);
  const int64_t id = blockIdx.x;
  int64_t grp;
  int qtile;
  if (p.order_kind == kOrderUnits) {
    const int u = p.order[id];             // the grid has order_n workgroups
    if (u == kNoUnit) return;
    grp = u / p.qtiles;
    qtile = u % p.qtiles;
  } else {
    const int64_t slot = id / kXcds;
    grp = (slot / p.qtiles) * kXcds + id % kXcds;
    if (grp >= p.groups) return;
    qtile = static_cast<int>(slot % p.qtiles);
  }
  const int64_t per_split = static_cast<int64_t>(p.batch) * p.num_kv_heads;
  const int split = static_cast<int>(grp / per_split);
  const int64_t rg = grp % per_split;
  const int rank = static_cast<int>(rg / p.num_kv_heads);
  const int g = static_cast<int>(rg % p.num_kv_heads);
  const int b = (p.order_kind == kOrderSeqs && rank < p.order_n) ? p.order[rank] : rank;
  if (p.gate && gate == 0) return;

  const int G = p.group;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // Workgroup-wide OR of a per-thread flag.  With five tile buffers it goes
  // through one word per wave at the start of the fifth (the library's own
  // reduction would need LDS beyond the buffers); the pipelined loop, that
  // buffer's only other user, loads into it after barriers that follow every
  // read here.
  auto wg_any = [&](bool v) -> bool {
    if constexpr (!PIPE) {
      return __syncthreads_or(v) != 0;
    } else {
      // (an LDS-typed pointer: a generic one made the compiler keep a 64-bit
      // address per word live across the key loop, and spill them)
      typedef __attribute__((address_space(3))) volatile int lds_word;
      lds_word *slot = (lds_word *)(lds4);
      const bool w = __builtin_amdgcn_ballot_w64(v) != 0;
      lds_barrier();       // earlier reads of the words are done
      if ((tid & 63) == 0) slot[wave] = w;
      lds_barrier();
      bool r = false;
#pragma unroll
      for (int i = 0; i < kWaves; ++i) r |= slot[i] != 0;
      return r;
    }
  };
  const int c = lane & 31;       // query column of this lane
  const int h = lane >> 5;       // which half of the 32x32 MFMA layout
  const int wrow = KS == 2 ? (wave % (kWaves / 2)) : wave;   // row slice of this wave
  const int kown = KS == 2 ? (wave / (kWaves / 2)) : 0;      // 32-key block of each tile (KS = 2)
  const int wv = __builtin_amdgcn_readfirstlane(wave);       // wave index as a scalar
  const int wpage = wv % 4;                                  // page of each tile this wave loads
  const int wpart = wv / 4;                                  // and which part of it
  const int kb = split * p.kv_chunk;

  // The reads below depend only on b and are issued together: the lengths,
  // the page of the first tile that this wave loads and, in lane j, the
  // window length of sequence j < b (the first 64 of those).  With a fixed
  // window, window_lens may be absent and prefix_lens is read in its place
  // and ignored.
  const bool fixed = p.fixed_window >= 0;
  const int32_t *wl = fixed ? p.prefix_lens : p.window_lens;
  const int32_t P_dev = load_now(p.prefix_lens + b);
  const int32_t W_dev = load_now(wl + b);
  const int32_t wl_lane = load_now(wl + min(lane, b));
  const int pid0 = wave_page(p, b, kb, wpage, std::true_type{});
  // lengths are clamped to the host-validated bounds, so a wrong device value
  // can give wrong numbers but never an access outside q, out or the workspace
  const int W = fixed ? p.fixed_window : min(max(W_dev, 0), p.max_window);
  const int P = min(max(P_dev, 0), p.max_prefix);
  const int M = G * W;
  const int row0 = qtile * kRowsPerTile;
  const int n_all = P + W;
  const int nsplit = min(p.splits, max(1, (n_all + p.kv_chunk - 1) / p.kv_chunk));
  // no rows in this query tile, or a split past the sequence's last
  if (row0 >= M || split >= nsplit) return;
  MBE_TL_REAL(1);

  // first query row of sequence b
  int cu = 0;
  if (fixed) {
    cu = b * p.fixed_window;
  } else {
    cu = lane < b ? min(max(wl_lane, 0), p.max_window) : 0;
    for (int j = lane + 64; j < b; j += 64) cu += min(max(p.window_lens[j], 0), p.max_window);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cu += __shfl_xor(cu, o);
    cu = __builtin_amdgcn_readfirstlane(cu);   // the same in every lane
  }

  // ---- this lane's two query rows (one per 32-row block of the wave), and
  // their Q^T operands in registers: lane (c, h) holds dims 16kk + 8h .. +7
  bool valid[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = row0 + wrow * kRowsPerWave + qb * 32 + c;
    valid[qb] = r < M && cu + r / G < p.total_q &&
                (!p.block_flags || p.block_flags[static_cast<int64_t>(b) * p.flag_stride + (r / G) / p.block_size]);
  }
  // index (cu + i) * Hq + hq of the output row of query block qb (row 0 for
  // an invalid lane); recomputed where needed rather than kept over the key
  // loop
  auto row_index = [&](int qb) -> int64_t {
    const int r = row0 + wrow * kRowsPerWave + qb * 32 + c;
    const int i = valid[qb] ? r / G : 0;
    const int hq = g * G + (valid[qb] ? r % G : 0);
    return static_cast<int64_t>(cu + i) * p.num_q_heads + hq;
  };
  // with block flags, a workgroup none of whose rows is flagged does nothing
  bool any_valid = false;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) any_valid |= valid[qb];
  if (p.block_flags && !wg_any(any_valid)) return;
  constexpr int KK = D / 16;
  bf16x8 qreg[QB][KK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (valid[qb])
        qreg[qb][kk] = *reinterpret_cast<const bf16x8 *>(p.q + row_index(qb) * D + kk * 16 + h * 8);
      else
        qreg[qb][kk] = bf16x8{};
    }

  // ---- key range of this split
  const int ke = min(n_all, kb + p.kv_chunk);
  int lim[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    int n = n_all;
    if (MODE == 1) {
      const int i = (row0 + wrow * kRowsPerWave + qb * 32 + c) / G;   // window position of the row
      n = min(n_all, P + (i / p.block_size + 1) * p.block_size);
    }
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

  // ---- loop-invariant LDS operand offsets of this lane
  constexpr int DB = D / 32;
  // K: row perm_row(c) (+32 for the second key block), chunk 2kk + h
  const int krow = perm_row(c);
  int koff[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) koff[kk] = krow * (2 * D) + (((2 * kk + h) ^ k_swz<D>(krow)) << 4);
  // V: page 2kbk + mm of the tile, dim c (+32 per dim block), keys 8h .. 8h+7
  // of the page (dims 32db + c and c share the half swap, 32 being a
  // multiple of 16)
  const int voff = Tile<D>::kKBytes + c * (kPageSize * 2) + (v_half(c, h) << 4);
  // Token-major V: transposing read q (q = 0, 1) of dim block db gives lane
  // (c, h) dim 32db + c at keys 8h + 4q .. +3 of a 16-key step: lane l reads
  // 4 dims (32db + 16((l >> 4) & 1) + 4(l & 3) ..) of key row 8h + (l & 15) / 4
  // (+ 4q), the 16 lanes of a group together a 4 x 16 block.
  int vtoff[DB];
  if constexpr (VT) {
    const int r = 8 * h + ((lane & 15) >> 2);                 // key row within the step, q = 0
    const int sw = v_swz<D>(r);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int chunk = 4 * db + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
      vtoff[db] = Tile<D>::kKBytes + r * (2 * D) + ((chunk ^ sw) << 4) + 8 * (lane & 1);
    }
  }

  f32x16 acc_o[QB][DB];
  float m_ref[QB];                       // reference, log2 units
  float l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_ref[qb] = kNegInf;
    l_run[qb] = 0.f;
  }

  // rows of this workgroup see keys [kb, lim); lim is smallest for the first
  // row, so tiles ending at or below it need no mask for any row
  int wg_min = ke;
  if (MODE == 1) wg_min = min(ke, P + ((row0 / G) / p.block_size + 1) * p.block_size);
  const int t_full = min(ntiles, max(0, (wg_min - kb) / kKeyTile));

  // K operands (A of S^T = K.Q^T) of 32-key block kbk
  auto read_k = [&](const char *buf, int kbk, bf16x8 (&a)[KK]) {
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) a[kk] = lds_read8(buf, koff[kk] + kbk * 32 * (2 * D));
  };
  // V operands (A of O^T += V^T.P^T) of 32-key block kbk
  auto read_v = [&](const char *buf, int kbk, bf16x8 (&va)[2][DB]) {
#pragma unroll
    for (int mm = 0; mm < 2; ++mm)
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        if constexpr (VT) {
          const char *at = buf + vtoff[db] + (2 * kbk + mm) * Tile<D>::kPageBytes;
          const bf16x4 lo = lds_read_tr4(at);
          const bf16x4 hi = lds_read_tr4(at + 4 * (2 * D));
          va[mm][db] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        } else {
          va[mm][db] = lds_read8(buf, voff + (2 * kbk + mm) * Tile<D>::kPageBytes + db * 32 * (kPageSize * 2));
        }
      }
  };
  // S^T of one 32-key block for both query blocks
  auto qk_mfma = [&](const bf16x8 (&a)[KK], f32x16 (&sc)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) sc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], qreg[qb][0], f32x16{}, 0, 0, 0);
#pragma unroll
    for (int kk = 1; kk < KK; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
        sc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], qreg[qb][kk], sc[qb], 0, 0, 0);
  };
  auto qk_block = [&](const char *buf, int kbk, f32x16 (&sc)[QB]) {
    bf16x8 a[KK];
    read_k(buf, kbk, a);
    qk_mfma(a, sc);
  };
  // keys at or past a row's limit get -inf
  // Element v of a lane holds key kblk0 + 8h + 16(v >> 3) + (v & 7).  With
  // token-major V the test is against the lane's room left, so each compare
  // takes a constant instead of one of 16 key offsets the compiler would
  // keep in registers (that kernel then needs no scratch; in the others the
  // same form makes the register allocation spill more, not less).
  auto mask_block = [&](int kblk0, f32x16 (&sc)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      if constexpr (VT) {
        int room = lim[qb] - kblk0 - 8 * h;
        asm volatile("" : "+v"(room));
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (16 * (v >> 3) + (v & 7) >= room) sc[qb][v] = kNegInf;
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kblk0 + 16 * (v >> 3) + 8 * h + (v & 7);
          if (key >= lim[qb]) sc[qb][v] = kNegInf;
        }
      }
    }
  };
  auto max_block = [&](f32x16 (&sc)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = kNegInf;
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[qb][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      m_ref[qb] = fmaxf(m_ref[qb], mx * p.scale_log2);
    }
  };
  // numerators 2^(s*scale*log2e - ref) to bf16 P^T, then O^T += V^T . P^T
  auto softmax_pv = [&](const bf16x8 (&va)[2][DB], f32x16 (&sc)[QB]) {
    bf16x8 pb[QB][2];   // [qb][m]: keys 16m + 8h .. +7 of this block
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float msafe = (m_ref[qb] == kNegInf) ? 0.f : m_ref[qb];
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][v], p.scale_log2, -msafe));
      // the row sum adds the bf16 numerators that enter P.V, two per dot2
      float lsum = l_run[qb];
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        const u32x4 w = {pack_bf16x2(e[8 * mm + 0], e[8 * mm + 1]), pack_bf16x2(e[8 * mm + 2], e[8 * mm + 3]),
                         pack_bf16x2(e[8 * mm + 4], e[8 * mm + 5]), pack_bf16x2(e[8 * mm + 6], e[8 * mm + 7])};
        pb[qb][mm] = __builtin_bit_cast(bf16x8, w);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          // (copied out first: a bit cast of the vector element w[k] itself
          // is compiled as a cast of w[0] by this compiler)
          const uint32_t wk = w[k];
          lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, wk), kOnes2, lsum, false);
        }
      }
      l_run[qb] = lsum;
    }
#pragma unroll
    for (int mm = 0; mm < 2; ++mm)
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          acc_o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[mm][db], pb[qb][mm], acc_o[qb][db], 0, 0, 0);
      }
  };
  // ---- key loop: tile t lives in buffer t % 4; tiles t+1..t+3 are in flight
  // while tile t is computed.  pid holds the page ids of the next tile to load.
  // Per-lane offsets of the direct loads, live for the whole kernel: a load's
  // address register is then never reused as the destination of an LDS read,
  // which would make the compiler wait for every load in flight first.
  uint32_t kload_off[Tile<D>::kWaveLoads];
  k_load_offsets<D>(kload_off, wpart);
  uint32_t vload_off;
  if constexpr (VT) vload_off = vt_load_offset<D>();
  else vload_off = (lane >> 1) * 32 + (v_half(lane >> 1, lane & 1) << 4);
  int pid = 0;                                             // this wave's page of the next tile
  auto buf_of = [&](int t) -> char * {
    switch (t & 3) {
      case 0: return lds0;
      case 1: return lds1;
      case 2: return lds2;
      default: return lds3;
    }
  };
  // direct loads of tile t into dst, then the page ids of tile t + 1
  auto issue = [&](int t, char *dst) {
    load_tile<D, VT>(p, g, wpage, wpart, pid, kload_off, vload_off, dst);
    pid = wave_page(p, b, kb + (t + 1) * kKeyTile, wpage);
  };
  // The same into buffer t % 4 with the buffer named at each call.  The
  // compiler tracks in-flight direct loads per LDS buffer only when it knows
  // the buffer; a load into a computed one would make every later LDS read,
  // the main loop's included, wait for all loads in flight.  (The asm
  // comments keep the four calls from being merged into one with a computed
  // destination.)
  auto issue_any = [&](int t) {
    switch (t & 3) {
      case 0: issue(t, lds0); asm volatile("; tile loads into buffer 0"); break;
      case 1: issue(t, lds1); asm volatile("; tile loads into buffer 1"); break;
      case 2: issue(t, lds2); asm volatile("; tile loads into buffer 2"); break;
      default: issue(t, lds3); asm volatile("; tile loads into buffer 3"); break;
    }
  };
  constexpr int kLoadsPerTile = 2 * Tile<D>::kWaveLoads; // direct loads per thread per tile
  // waits until at most n tiles' loads of this thread are still in flight,
  // then meets the other waves: afterwards every earlier tile is in LDS
  auto land = [&](int n) {
    if (n >= 2) __builtin_amdgcn_s_waitcnt(wait_vmcnt(2 * kLoadsPerTile));
    else if (n == 1) __builtin_amdgcn_s_waitcnt(wait_vmcnt(kLoadsPerTile));
    else __builtin_amdgcn_s_waitcnt(wait_vmcnt(0));
    lds_barrier();
  };
  // V rows of keys past n_all in tile t (only the last tile can have them)
  auto fix_tail = [&](int t) {
    const int key0 = kb + t * kKeyTile;
    if (key0 + kKeyTile > n_all) {
      zero_v_tail<D, VT>(buf_of(t), n_all - key0);
      lds_barrier();
    }
  };
  auto prologue = [&]() {
    pid = pid0;
    for (int t = 0; t < 3 && t < ntiles; ++t) issue_any(t);
    land(min(2, ntiles - 1));
    fix_tail(0);
  };
  auto compute = [&](const char *buf, int t, auto masked) {
    const int key0 = kb + t * kKeyTile;
    if constexpr (KS == 2) {
      f32x16 s0[QB];
      qk_block(buf, kown, s0);
      if constexpr (decltype(masked)::value) mask_block(key0 + 32 * kown, s0);
      bf16x8 va[2][DB];
      read_v(buf, kown, va);
      softmax_pv(va, s0);
    } else {
      f32x16 s0[QB], s1[QB];
      qk_block(buf, 0, s0);
      qk_block(buf, 1, s1);
      if constexpr (decltype(masked)::value) {
        mask_block(key0, s0);
        mask_block(key0 + 32, s1);
      }
      bf16x8 va[2][DB];
      read_v(buf, 0, va);
      softmax_pv(va, s0);
      read_v(buf, 1, va);
      softmax_pv(va, s1);
    }
  };
  // one tile through dynamically chosen buffers (remainder, masked tiles)
  auto generic_step = [&](int t, bool masked) {
    if (t + 3 < ntiles) issue_any(t + 3);
    if (masked) compute(buf_of(t), t, std::true_type{});
    else compute(buf_of(t), t, std::false_type{});
    if (t + 1 < ntiles) {
      land(min(2, ntiles - 2 - t));
      fix_tail(t + 1);
    }
  };

  // ---- software-pipelined key loop (KS = 1), by 32-key block n: the
  // scores of block n + 1 are computed on the matrix cores while block n's
  // scores, computed one half-step earlier, are exponentiated; then block
  // n's P.V.  Step t covers the two blocks of tile t, the second of which
  // scores the first block of tile t + 1.  Five buffers: at the top of step t
  // tiles t and t + 1 are in LDS and tiles t + 2, t + 3 in flight; step t
  // issues tile t + 4 into the buffer of tile t - 1, which every wave
  // finished reading before the barrier that ended step t - 1, and its own
  // barrier lands tile t + 2.  Every LDS read of step t is of tile t or t + 1.
  //
  // numerators of one block to bf16 P^T (keys 16m + 8h .. +7), row sums of
  // the bf16 numerators
  auto softmax_blk = [&](const f32x16 (&s)[QB], bf16x8 (&pb)[2]) {
    const float msafe = (m_ref[0] == kNegInf) ? 0.f : m_ref[0];
    float e[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) e[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[0][v], p.scale_log2, -msafe));
    float lsum = l_run[0];
#pragma unroll
    for (int mm = 0; mm < 2; ++mm) {
      const u32x4 w = {pack_bf16x2(e[8 * mm + 0], e[8 * mm + 1]), pack_bf16x2(e[8 * mm + 2], e[8 * mm + 3]),
                       pack_bf16x2(e[8 * mm + 4], e[8 * mm + 5]), pack_bf16x2(e[8 * mm + 6], e[8 * mm + 7])};
      pb[mm] = __builtin_bit_cast(bf16x8, w);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t wk = w[k];
        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, wk), kOnes2, lsum, false);
      }
    }
    l_run[0] = lsum;
  };
  // O^T += V^T . P^T for one block
  auto pv_mfma = [&](const bf16x8 (&va)[2][DB], const bf16x8 (&pb)[2]) {
#pragma unroll
    for (int mm = 0; mm < 2; ++mm)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        acc_o[0][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[mm][db], pb[mm], acc_o[0][db], 0, 0, 0);
  };
  // half-step for block n = block kbk of the tile in vbuf: s holds its
  // scores on entry and those of block n + 1 (block nkbk of the tile in
  // nbuf, first key nkey0) on exit
  auto half_step = [&](const char *vbuf, int kbk, const char *nbuf, int nkbk, int nkey0, f32x16 (&s)[QB],
                       auto masked) {
    bf16x8 va[2][DB];
    read_v(vbuf, kbk, va);
    f32x16 sn[QB];
    qk_block(nbuf, nkbk, sn);
    if constexpr (decltype(masked)::value) mask_block(nkey0, sn);
    bf16x8 pb[2];
    softmax_blk(s, pb);
    pv_mfma(va, pb);
    s[0] = sn[0];
  };
  auto pipe_step = [&](const char *vbuf, const char *kbuf, int t, f32x16 (&s)[QB], auto masked) {
    const int key0 = kb + t * kKeyTile;
    half_step(vbuf, 0, vbuf, 1, key0 + 32, s, masked);
    half_step(vbuf, 1, kbuf, 0, key0 + kKeyTile, s, masked);
  };
  auto pipe_last = [&](const char *vbuf, int t, f32x16 (&s)[QB]) {
    half_step(vbuf, 0, vbuf, 1, kb + t * kKeyTile + 32, s, std::true_type{});
    bf16x8 va[2][DB];
    read_v(vbuf, 1, va);
    bf16x8 pb[2];
    softmax_blk(s, pb);
    pv_mfma(va, pb);
  };
  // buffer t % 5 named at each use (see issue_any)
  auto buf5 = [&](int t) -> char * {
    switch (t % 5) {
      case 0: return lds0;
      case 1: return lds1;
      case 2: return lds2;
      case 3: return lds3;
      default: return lds4;
    }
  };
  auto issue5 = [&](int t) {
    switch (t % 5) {
      case 0: issue(t, lds0); asm volatile("; tile loads into buffer 0"); break;
      case 1: issue(t, lds1); asm volatile("; tile loads into buffer 1"); break;
      case 2: issue(t, lds2); asm volatile("; tile loads into buffer 2"); break;
      case 3: issue(t, lds3); asm volatile("; tile loads into buffer 3"); break;
      default: issue(t, lds4); asm volatile("; tile loads into buffer 4"); break;
    }
  };
  auto fix_tail5 = [&](int t) {
    const int key0 = kb + t * kKeyTile;
    if (key0 + kKeyTile > n_all) {
      zero_v_tail<D, VT>(buf5(t), n_all - key0);
      lds_barrier();
    }
  };
  auto pipelined_run = [&](bool set_ref) {
    pid = pid0;
    for (int t = 0; t < 4 && t < ntiles; ++t) issue5(t);
    land(min(2, max(0, ntiles - 2)));    // tiles 0 and 1
    fix_tail(0);
    if (ntiles > 1) fix_tail(1);
    MBE_TL_REAL(2);
    // the first block's scores; in the first run they give the reference
    f32x16 s[QB];
    qk_block(lds0, 0, s);
    if (t_full == 0) mask_block(kb, s);
    if (set_ref) max_block(s);
#pragma unroll
    for (int db = 0; db < DB; ++db) acc_o[0][db] = f32x16{};
    l_run[0] = 0.f;
    int t = 0;
    // five steps per iteration through fixed buffers; the blocks scored here
    // need no mask and every tile issued here exists
    for (; t + 8 < ntiles && t + 5 < t_full; t += 5) {
      issue(t + 4, lds4);
      pipe_step(lds0, lds1, t, s, std::false_type{});
      land(2);
      issue(t + 5, lds0);
      pipe_step(lds1, lds2, t + 1, s, std::false_type{});
      land(2);
      issue(t + 6, lds1);
      pipe_step(lds2, lds3, t + 2, s, std::false_type{});
      land(2);
      issue(t + 7, lds2);
      pipe_step(lds3, lds4, t + 3, s, std::false_type{});
      land(2);
      issue(t + 8, lds3);
      pipe_step(lds4, lds0, t + 4, s, std::false_type{});
      land(2);
    }
    for (; t < ntiles; ++t) {
      if (t + 4 < ntiles) issue5(t + 4);
      if (t + 1 == ntiles) pipe_last(buf5(t), t, s);
      else if (t + 1 >= t_full) pipe_step(buf5(t), buf5(t + 1), t, s, std::true_type{});
      else pipe_step(buf5(t), buf5(t + 1), t, s, std::false_type{});
      if (t + 2 < ntiles) {
        land(min(2, ntiles - 3 - t));
        fix_tail5(t + 2);
      }
    }
    lds_barrier();      // all waves done with the buffers
  };

  // Run 0 takes the reference from the first 32-key block.  Run 1 happens
  // only if some row sum left the safe range: it first finds the true row
  // maxima with a K.Q-only pass, then repeats the full pass.
  for (int run = 0; run < 2; ++run) {
    if constexpr (PIPE) {
      if (run == 1 && ntiles > 0) {
        // the true row maxima, from a scores-only pass
        m_ref[0] = kNegInf;
        prologue();
        for (int t = 0; t < ntiles; ++t) {
          if (t + 3 < ntiles) issue_any(t + 3);
          const char *buf = buf_of(t);
          const int key0 = kb + t * kKeyTile;
          f32x16 s0[QB], s1[QB];
          qk_block(buf, 0, s0);
          qk_block(buf, 1, s1);
          mask_block(key0, s0);
          mask_block(key0 + 32, s1);
          max_block(s0);
          max_block(s1);
          if (t + 1 < ntiles) {
            land(min(2, ntiles - 2 - t));
            fix_tail(t + 1);
          }
        }
        lds_barrier();
      }
      if (ntiles > 0) pipelined_run(run == 0);
      else {
        l_run[0] = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc_o[0][db] = f32x16{};
      }
      if (run == 1) break;
      bool bad = false;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float lt = l_run[qb] + __shfl_xor(l_run[qb], 32);
        bad |= valid[qb] && !(lt <= kSumLimit);
      }
      if (!wg_any(bad)) break;
    } else {
    if (ntiles > 0) {
      if (run == 1) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) m_ref[qb] = kNegInf;
        prologue();
        for (int t = 0; t < ntiles; ++t) {
          if (t + 3 < ntiles) issue_any(t + 3);
          const char *buf = buf_of(t);
          const int key0 = kb + t * kKeyTile;
          f32x16 s0[QB], s1[QB];
          qk_block(buf, 0, s0);
          qk_block(buf, 1, s1);
          mask_block(key0, s0);
          mask_block(key0 + 32, s1);
          max_block(s0);
          max_block(s1);
          if (t + 1 < ntiles) {
            land(min(2, ntiles - 2 - t));
            fix_tail(t + 1);
          }
        }
        lds_barrier();
      }
      prologue();
      if (run == 0) MBE_TL_REAL(2);
      if (run == 0) {
        f32x16 sc[QB];
        qk_block(lds0, 0, sc);
        mask_block(kb, sc);
        max_block(sc);
      }
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int db = 0; db < DB; ++db) acc_o[qb][db] = f32x16{};
      l_run[qb] = 0.f;
    }
    int t = 0;
    // unmasked tiles, four per iteration through fixed buffers; every tile
    // loaded here exists, so two tiles stay in flight at each barrier
    for (; t + 6 < ntiles && t + 3 < t_full; t += 4) {
      issue(t + 3, lds3);
      compute(lds0, t, std::false_type{});
      land(2);
      issue(t + 4, lds0);
      compute(lds1, t + 1, std::false_type{});
      land(2);
      issue(t + 5, lds1);
      compute(lds2, t + 2, std::false_type{});
      land(2);
      issue(t + 6, lds2);
      compute(lds3, t + 3, std::false_type{});
      land(2);
    }
    for (; t < ntiles; ++t) generic_step(t, t >= t_full);
    if (ntiles > 0) lds_barrier();      // all waves done with the buffers

    if (run == 1) break;
    bool bad = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float lt = l_run[qb] + __shfl_xor(l_run[qb], 32);
      bad |= valid[qb] && !(lt <= kSumLimit);
    }
    if (!wg_any(bad)) break;
    }
  }
  MBE_TL_REAL(3);

  if constexpr (KS == 2) {
    // the waves of the second key block hand their partial O and row sums
    // (same reference) to the waves of the first through the tile buffers,
    // which no wave reads any more: row slice j's O goes to buffer 0 or 1
    // (as many slices per buffer as fit), its sums to buffer 2
    constexpr int kXoBytes = QB * DB * 16 * 64 * 4;
    constexpr int kSlicesPerBuf = Tile<D>::kBufBytes / kXoBytes;
    static_assert(kSlicesPerBuf >= 1 && kWaves / 2 <= 2 * kSlicesPerBuf, "row slices fit two buffers");
    float *xo = reinterpret_cast<float *>((wrow < kSlicesPerBuf ? lds0 : lds1) + (wrow % kSlicesPerBuf) * kXoBytes);
    float *xl = reinterpret_cast<float *>(lds2) + wrow * QB * 64;
    if (kown == 1) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) xo[((qb * DB + db) * 16 + v) * 64 + lane] = acc_o[qb][db][v];
        xl[qb * 64 + lane] = l_run[qb];
      }
    }
    lds_barrier();
    if (kown == 1) return;      // no barrier follows
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc_o[qb][db][v] += xo[((qb * DB + db) * 16 + v) * 64 + lane];
      l_run[qb] += xl[qb * 64 + lane];
    }
  }

  // ---- epilogue
  float l_tot[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) l_tot[qb] = l_run[qb] + __shfl_xor(l_run[qb], 32);

  if (nsplit == 1) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      if (!valid[qb]) continue;
      const float inv = l_tot[qb] > 0.f ? 1.f / l_tot[qb] : 0.f;
      uint16_t *orow = p.out + row_index(qb) * D;
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
    MBE_TL_END();
    return;
  }

  // split-KV: write this split's partial result (merged by the merge kernel)
  const int64_t split_stride = static_cast<int64_t>(p.total_q) * p.num_q_heads;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (!valid[qb]) continue;
    const int64_t rowidx = row_index(qb);
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
      *reinterpret_cast<float2 *>(pml) = make_float2(m_ref[qb], l_tot[qb]);
    }
  }
  MBE_TL_END();
}

// Split-KV merge, run after the main kernel when some sequence was split (the
// kernel boundary makes every partial result visible; no cross-workgroup
// fences inside the main kernel).  Block (x, b) merges items x*256 .. of
// sequence b, an item being kMergeDims dims of one (window row, query head):
//   M = max m_s,  O = sum 2^(m_s-M) O_s / sum 2^(m_s-M) l_s   (split order).
constexpr int kMergeDims = 8;   // dims per merge thread: two 16-byte loads per split, one 16-byte store
template <int D>
__global__ __launch_bounds__(256) void window_attention_merge_kernel(AttnParams p) {
  // The gate, the lengths of b and, in lane j, the window length of sequence
  // j < b (the first 64 of those) are requested together; the partial sums
  // follow once the split count is known.  With a fixed window, window_lens
  // may be absent and prefix_lens is read in its place and ignored.
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const bool fixed = p.fixed_window >= 0;
  const int32_t *wl = fixed ? p.prefix_lens : p.window_lens;
  const int32_t gate = load_now(p.gate ? p.gate : p.prefix_lens);
  const int32_t P_dev = load_now(p.prefix_lens + b);
  const int32_t W_dev = load_now(wl + b);
  const int32_t wl_lane = load_now(wl + min(lane, b));
  if (p.gate && gate == 0) return;
  const int P = min(max(P_dev, 0), p.max_prefix);
  const int W = fixed ? p.fixed_window : min(max(W_dev, 0), p.max_window);
  const int n_all = P + W;
  const int nsplit = min(p.splits, max(1, (n_all + p.kv_chunk - 1) / p.kv_chunk));
  if (nsplit == 1) return;                  // written directly by the main kernel
  constexpr int DI = D / kMergeDims;
  const int64_t items = static_cast<int64_t>(W) * p.num_q_heads * DI;
  const int64_t item = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  // first query row of sequence b: the window lengths before it, summed
  // across the lanes of the wave (before any lane leaves)
  int cu = 0;
  if (fixed) {
    cu = b * p.fixed_window;
  } else {
    cu = lane < b ? min(max(wl_lane, 0), p.max_window) : 0;
    for (int j = lane + 64; j < b; j += 64) cu += min(max(p.window_lens[j], 0), p.max_window);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cu += __shfl_xor(cu, o);
  }
  if (item >= items) return;
  const int64_t r = item / DI;              // (window row, query head) within the sequence
  const int d0 = static_cast<int>(item % DI) * kMergeDims;
  if (cu + r / p.num_q_heads >= p.total_q) return;
  if (p.block_flags &&
      !p.block_flags[static_cast<int64_t>(b) * p.flag_stride + (r / p.num_q_heads) / p.block_size])
    return;                                 // row of an unflagged block: not written
  const int64_t rowidx = static_cast<int64_t>(cu) * p.num_q_heads + r;
  const int64_t split_stride = static_cast<int64_t>(p.total_q) * p.num_q_heads;
  // Every split below nsplit wrote this row (zeros and a -inf reference when
  // it saw none of its keys).  Splits are read in chunks of C = 8, 4, 2 or 1
  // (the smallest that holds what is left, at most 8; chunks of 16 would hold
  // twice the registers and halve the waves a SIMD keeps), all loads of a
  // chunk issued together (past nsplit the last split is read again and
  // weighted 0); the running maximum M and the sums are rescaled when a chunk
  // raises M.  With at most 8 splits this is exactly the two-step form
  // (M first, then the sums in split order).
  float mrun = kNegInf, lsum = 0.f;
  constexpr int Q = kMergeDims / 4;         // 16-byte loads per split
  float o[kMergeDims] = {};
  auto chunk = [&](int s0, auto csize) {
    constexpr int C = decltype(csize)::value;
    const int n = min(C, nsplit - s0);
    float2 ml[C];
    float4 po[C][Q];
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int64_t sp = s0 + min(j, n - 1);
      ml[j] = *reinterpret_cast<const float2 *>(p.part_ml + (sp * split_stride + rowidx) * 2);
#pragma unroll
      for (int q = 0; q < Q; ++q)
        po[j][q] = *reinterpret_cast<const float4 *>(p.part_o + (sp * split_stride + rowidx) * D + d0 + 4 * q);
    }
    // every load of the chunk is issued before any is used (the scheduler
    // would otherwise interleave them with the sums to save registers)
    __builtin_amdgcn_sched_barrier(0);
    float cmax = mrun;
#pragma unroll
    for (int j = 0; j < C; ++j)
      if (j < n) cmax = fmaxf(cmax, ml[j].x);
    // old sums to the new maximum (nothing to rescale while M is -inf)
    const float rescale = mrun == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mrun - cmax);
    lsum *= rescale;
#pragma unroll
    for (int i = 0; i < kMergeDims; ++i) o[i] *= rescale;
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const float wgt = (j < n && ml[j].x != kNegInf) ? __builtin_amdgcn_exp2f(ml[j].x - cmax) : 0.f;
      lsum += wgt * ml[j].y;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        o[4 * q + 0] += wgt * po[j][q].x;
        o[4 * q + 1] += wgt * po[j][q].y;
        o[4 * q + 2] += wgt * po[j][q].z;
        o[4 * q + 3] += wgt * po[j][q].w;
      }
    }
    mrun = cmax;
  };
  for (int s0 = 0; s0 < nsplit;) {
    const int left = nsplit - s0;
    if (left > 4) { chunk(s0, std::integral_constant<int, 8>{}); s0 += 8; }
    else if (left > 2) { chunk(s0, std::integral_constant<int, 4>{}); s0 += 4; }
    else if (left == 2) { chunk(s0, std::integral_constant<int, 2>{}); s0 += 2; }
    else { chunk(s0, std::integral_constant<int, 1>{}); s0 += 1; }
  }
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  uint4 st;
  st.x = pack_bf16x2(o[0] * inv, o[1] * inv);
  st.y = pack_bf16x2(o[2] * inv, o[3] * inv);
  st.z = pack_bf16x2(o[4] * inv, o[5] * inv);
  st.w = pack_bf16x2(o[6] * inv, o[7] * inv);
  *reinterpret_cast<uint4 *>(p.out + rowidx * D + d0) = st;
}

template <int D, int MODE>
hipError_t launch_t(const AttnParams &p, hipStream_t stream) {
  const int64_t grid = p.order_kind == kOrderUnits ? p.order_n : p.slots_per_xcd * kXcds;
  const dim3 g(static_cast<unsigned>(grid)), blk(kT);
  if (p.v_token_major) {
    if (p.key_split == 2) hipLaunchKernelGGL((window_attention_kernel<D, MODE, 2, 1, 0>), g, blk, 0, stream, p);
    else hipLaunchKernelGGL((window_attention_kernel<D, MODE, 1, 1, 0>), g, blk, 0, stream, p);
  } else {
    if (p.key_split == 2) hipLaunchKernelGGL((window_attention_kernel<D, MODE, 2, 0, 0>), g, blk, 0, stream, p);
    else if (p.pipelined) hipLaunchKernelGGL((window_attention_kernel<D, MODE, 1, 0, 1>), g, blk, 0, stream, p);
    else hipLaunchKernelGGL((window_attention_kernel<D, MODE, 1, 0, 0>), g, blk, 0, stream, p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;
  const int64_t items = static_cast<int64_t>(p.max_window) * p.num_q_heads * (D / kMergeDims);
  const dim3 mgrid(static_cast<unsigned>((items + 255) / 256), static_cast<unsigned>(p.batch));
  hipLaunchKernelGGL((window_attention_merge_kernel<D>), mgrid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_window_attention(const AttnParams &p, int head_dim, int mask_mode, hipStream_t stream) {
  if (head_dim == 128) return mask_mode == 1 ? launch_t<128, 1>(p, stream) : launch_t<128, 0>(p, stream);
  return mask_mode == 1 ? launch_t<64, 1>(p, stream) : launch_t<64, 0>(p, stream);
}

}  // namespace mbe

#ifdef MBE_TIMELINE
// Profiling builds only: copy out / clear the phase timeline of the last
// attention launches (8 unsigned 64-bit entries per workgroup, the first
// 8192 workgroups).  Return a hipError_t code.
extern "C" int mbe_timeline_read(void *dst, size_t bytes) {
  if (bytes > sizeof(mbe::g_timeline)) bytes = sizeof(mbe::g_timeline);
  return static_cast<int>(hipMemcpyFromSymbol(dst, HIP_SYMBOL(mbe::g_timeline), bytes, 0, hipMemcpyDeviceToHost));
}
extern "C" int mbe_timeline_clear(void) {
  void *ptr = nullptr;
  hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(mbe::g_timeline));
  if (e == hipSuccess) e = hipMemset(ptr, 0, sizeof(mbe::g_timeline));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  return static_cast<int>(e);
}
#endif
