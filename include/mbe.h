/*
 * mbe.h -- C ABI of libmbe: the editing-pass hot path of Multi-Block Editing
 * (MBE) for block-diffusion language models, for AMD MI355X (gfx950).
 *
 * Paper: "Beyond Block Boundaries: Multi-Block Editing for Diffusion Large
 * Language Models".
 *
 * Conventions shared by every call
 *   - Every buffer argument is device memory owned by the caller.  The library
 *     keeps no pointer after a call returns and allocates nothing.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream).  They never synchronise; results are valid once the stream has
 *     been synchronised.  Kernels are launched on the current HIP device;
 *     every buffer and the stream must belong to it.
 *   - Arguments are validated on the host before any HIP call.  A failed
 *     check returns a non-OK status, launches nothing and writes nothing.
 *     mbe_last_error() then holds a thread-local description.
 *   - Per-sequence values that live in device memory (page ids, lengths) are
 *     preconditions and are not read back.  The attention calls clamp page
 *     ids outside [0, num_pages) into range, so a bad table gives wrong
 *     numbers but never an out-of-bounds access; the KV write-back skips a
 *     token whose table slot or page id is out of range instead of writing
 *     it anywhere else.  With the environment variable MBE_DEBUG_CHECK=1, the
 *     attention calls and mbe_kv_write copy the lengths and the page table to
 *     the host (on the call's stream, then synchronising it) and return
 *     MBE_ERR_BAD_VALUE on a violation; calls made while the stream is being
 *     captured into a graph are not checked.
 *   - An error from the HIP runtime is returned as MBE_ERR_HIP, with the HIP
 *     error string in mbe_last_error().
 *   - No global mutable state except the thread-local error string.  Calls
 *     that share a workspace must not overlap in time.
 *   - The attention and edit-selection calls launch one kernel, plus a small
 *     merge/finalize kernel when the work is split across workgroups (see the
 *     workspace sizes).  mbe_threshold_update adds one per-block kernel.
 */
#ifndef MBE_H_
#define MBE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MBE_OK = 0,
  MBE_ERR_NULL_ARG = 1,     /* a required pointer is NULL                      */
  MBE_ERR_BAD_SHAPE = 2,    /* sizes inconsistent or negative                  */
  MBE_ERR_UNSUPPORTED = 3,  /* head_dim, page size or mask mode not supported  */
  MBE_ERR_WORKSPACE = 4,    /* workspace missing or smaller than required      */
  MBE_ERR_HIP = 5,          /* HIP runtime or launch error                     */
  MBE_ERR_BAD_VALUE = 6     /* bad scalar (NaN threshold) or, under
                               MBE_DEBUG_CHECK=1, a bad per-sequence value     */
} mbe_status;

/* Attention scope of the window queries.
 *   MBE_MASK_WINDOW_BIDIR: every prefix token and every window token is
 *     visible.  This is the MBE editing pass, with full attention within the
 *     window W_j = [j*B, (j+1)B) (paper, Sec. "Training-Free MBE Decoding",
 *     Eq. (4)).
 *   MBE_MASK_BLOCK_CAUSAL: every prefix token and the window blocks up to the
 *     query's own block are visible.  This is the standard block-diffusion
 *     scope (Sec. "Block diffusion") that refresh recomputes use.
 * The two coincide when the window is one block. */
typedef enum { MBE_MASK_WINDOW_BIDIR = 0, MBE_MASK_BLOCK_CAUSAL = 1 } mbe_mask_mode;

/* Layout of the V pages (K pages are always token-major). */
typedef enum {
  MBE_V_TOKEN_MINOR = 0,  /* v_pages[num_pages][num_kv_heads][head_dim][16]             */
  MBE_V_TOKEN_MAJOR = 1   /* v_pages[num_pages][num_kv_heads][16][head_dim], like K: the
                             common paged-cache layout                                  */
} mbe_v_layout;

/* Paged KV cache for one layer.  Pages hold 16 tokens; all bf16.
 *   k_pages: [num_pages][num_kv_heads][16][head_dim]   token-major page
 *   v_pages: as v_layout says (token-minor [head_dim][16] or token-major
 *            [16][head_dim] per page and head)
 * Token t of sequence b is slot t % 16 of page page_table[b][t / 16].  The
 * window's own K/V (tokens P_b .. P_b+W_b-1) are read through the same table
 * from pages the caller provides.  The library only reads the cache, as the
 * paper's cache control requires (Sec. "Infrastructure Optimization").
 * The bytes of token slots that no sequence covers (the tail of a sequence's
 * last page) are never used and may hold anything, NaN included. */
typedef struct {
  const void *k_pages;
  const void *v_pages;
  int32_t num_pages;
  int32_t page_size;     /* must be 16            */
  int32_t num_kv_heads;  /* Hkv >= 1              */
  int32_t head_dim;      /* D: 64 or 128          */
  int32_t v_layout;      /* mbe_v_layout (0 = token-minor)  */
} mbe_paged_kv;

/* Options of the attention calls.  The bounds are host-side facts the caller
 * knows without reading device memory.  They size the grid and the
 * workspace; the kernels read the true lengths from device memory. */
typedef struct {
  int32_t batch;              /* number of sequences, >= 0                          */
  int32_t num_q_heads;        /* Hq, a multiple of num_kv_heads                      */
  int32_t max_pages_per_seq;  /* row length of page_table                           */
  int32_t total_q;            /* rows of q/out = sum of window lengths               */
  int32_t max_prefix_len;     /* >= every P_b                                        */
  int32_t max_window_len;     /* >= every W_b; a multiple of block_size              */
  int32_t mask_mode;          /* mbe_mask_mode                                      */
  float softmax_scale;        /* <= 0 selects 1/sqrt(head_dim)                      */
  int32_t kv_split_tokens;    /* keys per split-KV chunk; 0 lets the library choose;
                                 otherwise a positive multiple of 64                 */
  const int32_t *host_prefix_lens;  /* optional HOST copies of prefix_lens /         */
  const int32_t *host_window_lens;  /* window_lens ([batch] each, NULL = unknown).
                                 They are read on the host only, to size the
                                 split-KV chunks from the total work and to start
                                 the longest sequences first; they must equal the
                                 device values.  Ignored when batch > 1024.          */
  void *workspace;            /* device memory of at least
                                 mbe_window_attention_workspace_size bytes
                                 (mbe_block_diffusion_workspace_size for
                                 block_diffusion_attention), 256-byte aligned, any
                                 contents (split-KV partial results); may be NULL
                                 when that size is 0                                 */
  size_t workspace_bytes;
  void *stream;               /* hipStream_t                                        */
  const uint8_t *block_flags; /* optional DEVICE uint8 [batch][max_window_len /
                                 block_size] (NULL = every row).  The rows of window
                                 block i of sequence b (positions i*B .. i*B+B-1)
                                 are computed and written only when
                                 block_flags[b * (max_window_len / block_size) + i]
                                 is nonzero; the other rows of out are left as they
                                 were.  This is the targeted refresh: recompute
                                 only the blocks an editing pass changed (paper,
                                 Sec. "Infrastructure Optimization", cache control).
                                 block_diffusion_attention reads one flag per
                                 sequence ([batch][1]).                             */
  const int32_t *run_if_nonzero; /* optional DEVICE int32 (NULL = always run).  When
                                 it holds 0 when the call runs on the stream, the
                                 call computes and writes nothing.  With the changed
                                 count of the previous editing pass, a sequence of
                                 at most N_MBE passes captured in one graph stops
                                 early without a host round trip (paper, Sec.
                                 "Training-Free MBE Decoding", the pass loop).      */
} mbe_attn_opts;

/* Editing-window attention (paper, Sec. "Training-Free MBE Decoding", Eq. (4)).
 *   q:           bf16 [total_q][Hq][D]; the W_b rows of sequence b start at row
 *                sum_{b' < b} W_b' and row i is window position P_b + i.
 *   paged_kv:    the cache, see mbe_paged_kv.
 *   page_table:  int32 [batch][max_pages_per_seq]; must cover P_b + W_b tokens.
 *   prefix_lens: int32 [batch], P_b >= 0 committed prefix tokens.
 *   window_lens: int32 [batch], W_b >= 0, a multiple of block_size.
 *   block_size:  B >= 1.
 *   out:         bf16 [total_q][Hq][D], written for every row.
 * Query head h reads KV head h / (Hq / Hkv).  The scale is applied to q.k
 * before a softmax over the visible keys (fp32 accumulation).
 * Returns MBE_OK with no launch when batch or total_q is 0. */
mbe_status mbe_window_attention(const void *q, const mbe_paged_kv *paged_kv,
                                const int32_t *page_table, const int32_t *prefix_lens,
                                const int32_t *window_lens, int32_t block_size, void *out,
                                const mbe_attn_opts *opts);

/* Standard single-block block-diffusion attention (paper, Sec. "Block
 * diffusion"): each sequence's B = block_size queries attend to its prefix
 * and bidirectionally to their own block.  This is mbe_window_attention with
 * W_b = block_size for every b; opts->max_window_len and opts->mask_mode are
 * ignored, and opts->total_q must equal batch * block_size. */
mbe_status block_diffusion_attention(const void *q, const mbe_paged_kv *paged_kv,
                                     const int32_t *page_table, const int32_t *prefix_lens,
                                     int32_t block_size, void *out, const mbe_attn_opts *opts);

/* Workspace bytes mbe_window_attention needs for these shapes and options
 * (all of opts, host lengths included, since they shape the split plan): the
 * split-KV partial results.  0 means the plan needs no split and no
 * workspace.  When some sequence is split, the call runs a second, small
 * kernel that merges the partial results.  The plan does not depend on the
 * block size; the call itself checks that max_window_len is a multiple of it.
 * Returns (size_t)-1 if the arguments are invalid. */
size_t mbe_window_attention_workspace_size(const mbe_paged_kv *paged_kv, const mbe_attn_opts *opts);

/* Launch plan of mbe_window_attention for these shapes and options, made on
 * the host exactly as the call makes it (no device access): for profiling
 * tools and tuning.  Not needed to run the call. */
typedef struct {
  int32_t splits;       /* key-range splits per sequence (1 = no split-KV merge) */
  int32_t kv_chunk;     /* keys per split                                        */
  int32_t key_split;    /* 2: two waves share every key tile of one row block    */
  int32_t pipelined;    /* 1: the software-pipelined key loop                    */
  int64_t workgroups;   /* grid size of the main kernel                          */
} mbe_attn_plan;

/* Fills *plan; returns MBE_OK, or an error status (and leaves *plan alone)
 * when the arguments are invalid, as mbe_window_attention_workspace_size
 * would return (size_t)-1. */
mbe_status mbe_window_attention_plan(const mbe_paged_kv *paged_kv, const mbe_attn_opts *opts, mbe_attn_plan *plan);

/* Workspace bytes block_diffusion_attention needs for these shapes and
 * options.  Its split plan takes W_b = block_size for every sequence (and
 * the host prefix lengths when given), so it can differ from
 * mbe_window_attention_workspace_size with the same opts.
 * Returns (size_t)-1 if the arguments are invalid. */
size_t mbe_block_diffusion_workspace_size(const mbe_paged_kv *paged_kv,
                                          const mbe_attn_opts *opts, int32_t block_size);

/* Confidence-based edit selection (paper, Sec. "Configurable threshold
 * decoding", Eq. (1), the token-to-token set), for every row r:
 *   a       = lowest index v with logits[r][v] maximal
 *   conf[r] = softmax probability of a = 1 / sum_v exp(logits[r][v] - logits[r][a])
 *   changed = (a != cur_tokens[r]) && (conf[r] >= threshold)
 *   new_tokens[r] = changed ? a : cur_tokens[r];  changed_mask[r] = changed
 * logits: bf16 [rows][row_stride], row_stride >= vocab; -inf entries allowed;
 * NaN or all -inf rows are outside the contract.  Accumulation is fp32; conf
 * is a correctly rounded reciprocal.  Deterministic: the same inputs give
 * bitwise the same outputs.  workspace: mbe_edit_select_workspace_size bytes,
 * 256-byte aligned, any contents (per-chunk partial results when a row is
 * reduced by several workgroups; may be NULL when the size is 0).
 * Returns MBE_OK with no launch when rows is 0; MBE_ERR_BAD_VALUE for a NaN
 * threshold. */
mbe_status mbe_edit_select(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                           const int32_t *cur_tokens, float threshold, int32_t *new_tokens,
                           float *conf, uint8_t *changed_mask, void *workspace,
                           size_t workspace_bytes, void *stream);

/* Workspace bytes mbe_edit_select needs for rows x vocab (0 = none).
 * Returns (size_t)-1 for negative sizes. */
size_t mbe_edit_select_workspace_size(int64_t rows, int64_t vocab);

/* ---------------------------------------------------------------------------
 * Full threshold update (paper, Sec. "Configurable threshold decoding",
 * Eq. (1) and the force-unmask rule after it).  Rows form blocks of
 * block_size consecutive rows (row r belongs to block r / block_size).  With
 * a = lowest index of the row maximum and conf[r] its softmax probability (as
 * in mbe_edit_select), each row gets an action:
 *   MBE_UNMASK        cur == mask_id and conf > omega_mask          (Gamma_t)
 *   MBE_FORCE_UNMASK  cur == mask_id, no row of its block is MBE_UNMASK, and
 *                     it has the highest conf among the block's masked rows
 *                     (the lowest such row on ties)
 *   MBE_EDIT          cur != mask_id, a != cur and conf >= omega_edit (Delta_t,
 *                     the edit rule of mbe_edit_select)
 *   MBE_KEEP          otherwise
 * new_tokens[r] = a for every action but MBE_KEEP, cur otherwise.
 * block_changed[k] = 1 when some row of block k has an action other than
 * MBE_KEEP.  changed_count (device int32, may be NULL) receives the number of
 * such rows, so a loop of editing passes can stop when it reaches 0 without
 * copying per-row results to the host.  entropy (may be NULL) receives each
 * row's softmax entropy in nats, -sum_v p_v ln p_v, computed in the same pass
 * over the logits (the input of the tail-entropy selection below).
 * run_if_nonzero (device int32, may be NULL): when it holds 0 the pass
 * changes nothing without reading the logits: every action is MBE_KEEP,
 * new_tokens = cur_tokens, block_changed = 0 and changed_count = 0, while
 * conf and entropy are left as they were.  Given the previous pass's
 * changed_count (a different buffer: the pass zeroes its own), the passes
 * after the first one that changes nothing cost about a launch each, with no
 * host read (paper, Sec. "Training-Free MBE Decoding": at most N_MBE passes,
 * stopping when no token changes).  new_tokens may be cur_tokens itself (an
 * in-place update).
 * rows must be a multiple of block_size.  logits/threshold contract as for
 * mbe_edit_select.  workspace: mbe_threshold_update_workspace_size bytes,
 * 256-byte aligned, any contents.  MBE_ERR_BAD_VALUE for a NaN threshold or
 * run_if_nonzero == changed_count. */
typedef enum { MBE_KEEP = 0, MBE_UNMASK = 1, MBE_FORCE_UNMASK = 2, MBE_EDIT = 3 } mbe_action;

mbe_status mbe_threshold_update(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                const int32_t *cur_tokens, int32_t mask_id, int32_t block_size,
                                float omega_mask, float omega_edit, int32_t *new_tokens, float *conf,
                                uint8_t *action, uint8_t *block_changed, int32_t *changed_count,
                                float *entropy, const int32_t *run_if_nonzero, void *workspace,
                                size_t workspace_bytes, void *stream);

/* Workspace bytes mbe_threshold_update needs (the per-row predictions plus
 * the per-chunk partials of mbe_edit_select).  (size_t)-1 for negative sizes. */
size_t mbe_threshold_update_workspace_size(int64_t rows, int64_t vocab);

/* mbe_threshold_update for callers that cannot allocate device memory and
 * hold no workspace (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and checks as
 * mbe_threshold_update, without the workspace: the scratch it needs (the
 * per-row predictions and chunk partials) lives in a static 1 MiB device
 * array inside the library, one per GPU, kept until the process ends.  Calls
 * whose scratch (mbe_threshold_update_workspace_size(rows, vocab)) exceeds
 * 1 MiB, i.e. beyond 262144 rows, return MBE_ERR_WORKSPACE and launch
 * nothing.  It calls no allocator.  All calls on one GPU share its array:
 * calls that overlap in time on one GPU (different streams or host threads)
 * race; calls on one stream are ordered and safe. */
mbe_status mbe_threshold_update_noalloc(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                        const int32_t *cur_tokens, int32_t mask_id, int32_t block_size,
                                        float omega_mask, float omega_edit, int32_t *new_tokens, float *conf,
                                        uint8_t *action, uint8_t *block_changed, int32_t *changed_count,
                                        float *entropy, const int32_t *run_if_nonzero, void *stream);

/* Tail-entropy score of every block (paper, Sec. "Training-Free MBE
 * Decoding", Eq. (5)): scores[k] = mean of the ceil(rho * block_size) largest
 * entropy values of rows k*block_size .. (k+1)*block_size - 1.  The values are
 * summed from the largest down, so the result does not depend on launch
 * shape.  1 <= block_size <= 1024 and 1 <= ceil(rho * block_size) <= block_size. */
mbe_status mbe_tail_entropy_scores(const float *entropy, int64_t num_blocks, int32_t block_size,
                                   float rho, float *scores, void *stream);

/* Start block of every sequence's editing window (Eq. (6)): with
 * j = current_block[b], start_block[b] = the block i in
 * [max(0, j - k_max + 1), j) with the highest scores[b * score_stride + i];
 * the earliest such block on ties (the widest window); j itself when j = 0.
 * current_block values are clamped to [0, score_stride]. */
mbe_status mbe_select_start_block(const float *scores, int32_t batch, int32_t score_stride,
                                  const int32_t *current_block, int32_t k_max, int32_t *start_block,
                                  void *stream);

/* Write-back of recomputed K/V (paper, Sec. "Infrastructure Optimization",
 * cache control: after editing, changed blocks are recomputed under standard
 * attention and their K/V restore the cache).  Token t < lens[b] of sequence
 * b (rows of sequence b start at sum_{b' < b} lens[b']) is written at
 * absolute position start_pos[b] + t, i.e. slot (position % 16) of page
 * page_table[b][position / 16], for every KV head:
 *   k_pages[page][head][slot][:] = k_new[row][head][:]      (bf16)
 *   v_pages[page][head][:][slot] = v_new[row][head][:]      (v_layout MBE_V_TOKEN_MINOR)
 *   v_pages[page][head][slot][:] = v_new[row][head][:]      (v_layout MBE_V_TOKEN_MAJOR)
 * k_new/v_new: bf16 [total_tokens][num_kv_heads][head_dim]; max_len bounds
 * every lens[b] (host-known, sizes the grid).  Other slots are not touched.
 * block_flags (device uint8, may be NULL = write every token): the targeted
 * refresh; token t of sequence b is written only when
 * block_flags[b * ceil(max_len / block_size) + t / block_size] is nonzero
 * (the row numbering of k_new/v_new does not change).  block_size >= 1 when
 * block_flags is given, ignored otherwise.
 * Preconditions (checked under MBE_DEBUG_CHECK=1): positions lie inside the
 * sequence's table row, page ids inside the pool, sum of lens = total_tokens.
 * A token that breaks them is not written (it never lands on another slot). */
mbe_status mbe_kv_write(void *k_pages, void *v_pages, int32_t num_pages, int32_t num_kv_heads,
                        int32_t head_dim, int32_t v_layout, const int32_t *page_table, int32_t max_pages_per_seq,
                        const int32_t *start_pos, const int32_t *lens, int32_t batch, int32_t max_len,
                        int32_t total_tokens, const void *k_new, const void *v_new,
                        const uint8_t *block_flags, int32_t block_size, void *stream);

/* Blocks to recompute after editing, from the per-block changed flags
 * ([batch][num_blocks], e.g. block_changed of mbe_threshold_update laid out
 * per sequence).  MBE_REFRESH_CHANGED: exactly the changed blocks, as the
 * paper describes.  MBE_REFRESH_CHANGED_AND_LATER: also every block after the
 * first changed one, whose standard-scope K/V attended to the old tokens. */
typedef enum { MBE_REFRESH_CHANGED = 0, MBE_REFRESH_CHANGED_AND_LATER = 1 } mbe_refresh_mode;

mbe_status mbe_refresh_blocks(const uint8_t *block_changed, int32_t batch, int32_t num_blocks,
                              int32_t mode, uint8_t *refresh, void *stream);

/* Static description of a status code. */
const char *mbe_status_string(mbe_status s);

/* Thread-local detail of the last non-OK status returned on this thread. */
const char *mbe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MBE_H_ */
