// Internal launch interface between the C ABI (abi.cpp) and the HIP kernels.
// Not installed; callers use include/mbe.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mbe.h"

namespace mbe {

// ---------------------------------------------------------------- attention
constexpr int kPageSize = 16;
constexpr int kKeyTile = 64;          // keys per LDS tile (4 pages)
constexpr int kRowsPerWave = 32;      // packed (window position, q head) rows per wave
constexpr int kWaves = 8;               // two per SIMD
constexpr int kRowsPerTile = kRowsPerWave * kWaves;   // rows per workgroup
constexpr int kXcds = 8;              // MI355X: workgroups go round-robin over 8 XCDs
constexpr int kMaxOrder = 1024;       // dispatch-order entries passed in the kernel arguments
constexpr uint16_t kNoUnit = 0xFFFF;  // dispatch-table slot without work



enum AttnOrderKind : int32_t { kOrderNone = 0, kOrderSeqs = 1, kOrderUnits = 2 };

struct AttnParams {
  const uint16_t *q;          // bf16 [total_q][Hq][D]
  const uint16_t *k_pages;    // bf16 [num_pages][Hkv][16][D]
  const uint16_t *v_pages;    // bf16 [num_pages][Hkv][D][16], or [num_pages][Hkv][16][D] when v_token_major
  const int32_t *page_table;  // [batch][max_pages]
  const int32_t *prefix_lens; // [batch]
  const int32_t *window_lens; // [batch] (unused when fixed_window >= 0)
  uint16_t *out;              // bf16 [total_q][Hq][D]
  float *part_o;              // fp32 [splits][total_q][Hq][D]   (split-KV only)
  float *part_ml;             // fp32 [splits][total_q][Hq][2]   (split-KV only)
  int32_t batch, num_q_heads, num_kv_heads, group, num_pages, max_pages;
  int32_t block_size, total_q, fixed_window;
  int32_t max_prefix, max_window;   // host-validated bounds; device lengths are clamped to them
  int32_t qtiles, splits, kv_chunk;
  int32_t key_split;          // 1, or 2 when a sequence has at most 128 rows per KV head
  int32_t v_token_major;      // V pages [16][D] (like K) instead of [D][16]
  int32_t pipelined;          // software-pipelined key loop (token-minor V, no key split)
  int64_t groups;             // (split, sequence rank, KV head) groups of qtiles work units
  int64_t slots_per_xcd;      // grid = kXcds * slots_per_xcd workgroups
  float scale_log2;           // softmax scale * log2(e)
  const uint8_t *block_flags; // [batch][flag_stride] or null: rows of unflagged window blocks are skipped
  int32_t flag_stride;
  const int32_t *gate;        // device int32 or null: the call does nothing when *gate == 0
  // Dispatch order, from the host lengths when given.
  //   kOrderSeqs:  order[rank] is the sequence of that rank (longest first);
  //                groups are dealt round-robin to the XCDs by formula.
  //   kOrderUnits: workgroup i < order_n runs work unit order[i] =
  //                grp * qtiles + query tile (kNoUnit: none), where
  //                grp = split * batch * Hkv + sequence * Hkv + KV head.
  //   kOrderNone:  natural sequence order, formula dealing.
  int32_t order_kind;
  int32_t order_n;
  uint16_t order[kMaxOrder];
};

hipError_t launch_window_attention(const AttnParams &p, int head_dim, int mask_mode,
                                   hipStream_t stream);

// ------------------------------------------------------------ edit selection
constexpr int kEsThreads = 256;
constexpr int kEsVecPerThread = 2;   // 16-byte loads per thread per iteration

struct EsPartial {
  float m;        // running max logit
  float s;        // sum of 2^y, y = (l - m) log2(e)
  int32_t idx;    // lowest index attaining m
  float t;        // sum of 2^y * y (entropy accumulator; 0 when not asked for)
};

// Row reduction (edit selection, or the first step of the threshold update).
struct EsParams {
  const uint16_t *logits;   // bf16 [rows][ld]
  int64_t rows, vocab, ld;
  int64_t chunk_len;        // elements per chunk, a multiple of 8
  int32_t chunks;           // chunks per row
  int32_t update;           // 0: edit selection decides; 1: write pred/conf/entropy only
  const int32_t *cur;
  float threshold;          // edit threshold (omega_edit for the update)
  int32_t *new_tokens;
  float *conf;
  uint8_t *changed;         // edit selection only
  EsPartial *partials;      // [rows][chunks]   (chunks > 1 only)
  // threshold update
  int32_t *pred;            // [rows] argmax (workspace)
  float *entropy;           // [rows] nats, or null
  int32_t *changed_count;   // zeroed by the row pass, or null
  uint8_t *action;          // [rows]
  uint8_t *block_changed;   // [rows / block_size]
  int32_t mask_id, block_size;
  float omega_mask;
  const int32_t *gate;      // threshold update: when *gate == 0 the pass changes nothing
};

void edit_select_plan(int64_t rows, int64_t vocab, int32_t *chunks, int64_t *chunk_len);
hipError_t launch_edit_select(const EsParams &p, bool vector_loads, hipStream_t stream);
hipError_t launch_threshold_update(const EsParams &p, bool vector_loads, hipStream_t stream);

// Tail-entropy scores, start-block choice, refresh flags, KV write-back.
hipError_t launch_tail_entropy_scores(const float *entropy, int64_t num_blocks, int32_t block_size, int32_t k,
                                      float *scores, hipStream_t stream);
hipError_t launch_select_start_block(const float *scores, int32_t batch, int32_t stride, const int32_t *current,
                                     int32_t k_max, int32_t *start, hipStream_t stream);
hipError_t launch_refresh_blocks(const uint8_t *changed, int32_t batch, int32_t num_blocks, int32_t mode,
                                 uint8_t *refresh, hipStream_t stream);

struct KvWriteParams {
  uint16_t *k_pages, *v_pages;
  int32_t num_pages, num_kv_heads, head_dim;
  int32_t v_token_major;           // V pool [page][head][16][D] like K, else [page][head][D][16]
  const int32_t *page_table;
  int32_t max_pages;
  const int32_t *start_pos, *lens;
  int32_t batch, max_len, total_tokens;
  const uint16_t *k_new, *v_new;   // bf16 [total_tokens][heads][D]
  const uint8_t *block_flags;      // [batch][flag_stride], or null: write every token
  int32_t block_size, flag_stride; // token t of a sequence is in block t / block_size
};
hipError_t launch_kv_write(const KvWriteParams &p, hipStream_t stream);

// ------------------------------------------------- shared by the C entry points
// Sets the thread-local error string; returns s.
mbe_status report(mbe_status s, const char *fmt, ...);
// Argument checks of the threshold update (all but the workspace); *need
// receives the workspace bytes the call uses (0 when rows == 0).
mbe_status threshold_update_check(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                  const int32_t *cur_tokens, int32_t block_size, float omega_mask, float omega_edit,
                                  const int32_t *new_tokens, const float *conf, const uint8_t *action,
                                  const uint8_t *block_changed, const int32_t *changed_count,
                                  const int32_t *run_if_nonzero, size_t *need);
// Launches a checked threshold update on a workspace of at least *need bytes.
mbe_status threshold_update_launch(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                   const int32_t *cur_tokens, int32_t mask_id, int32_t block_size, float omega_mask,
                                   float omega_edit, int32_t *new_tokens, float *conf, uint8_t *action,
                                   uint8_t *block_changed, int32_t *changed_count, float *entropy,
                                   const int32_t *run_if_nonzero, void *workspace, void *stream);


}  // namespace mbe
