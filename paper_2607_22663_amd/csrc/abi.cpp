// C ABI of libmbe: argument validation, split planning, workspace sizing and
// dispatch to the HIP kernels.  Every check runs before the first HIP call,
// so the validation paths work on a machine without a GPU.
#include "mbe.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <functional>
#include <string>
#include <vector>

#include "internal.h"

namespace {

thread_local std::string g_last_error;

mbe_status fail(mbe_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

mbe_status hip_fail(hipError_t e, const char *where) {
  return fail(MBE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool debug_checks() {
  const char *v = std::getenv("MBE_DEBUG_CHECK");
  return v && v[0] == '1';
}

// Key loop of the attention with token-minor V and no key split: the
// software-pipelined loop (scores of the next 32-key block on the matrix
// cores while this block is exponentiated, five LDS tile buffers) when a
// work unit spans at least kPipeMinTiles 64-key tiles; below that its longer
// start-up costs more than it saves (measured: long-context and 8-block
// windows over 16K prefixes gain 2%, 4-block windows and shorter loops lose
// up to 9%).  MBE_ATTN_PIPELINE=0 / 1 forces either loop (tests use it to
// run both on every shape).
constexpr int64_t kPipeMinTiles = 96;
int pipeline_override() {
  const char *v = std::getenv("MBE_ATTN_PIPELINE");
  if (v && v[0] == '0') return 0;
  if (v && v[0] == '1') return 1;
  return -1;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Split-KV plan for the attention calls, from host-known values only.
struct AttnPlan {
  int32_t group = 0, qtiles = 0, splits = 1, kv_chunk = 0;
  int64_t groups = 0, slots_per_xcd = 0;
  size_t part_o_off = 0, part_ml_off = 0, bytes = 0;
  int32_t order_kind = mbe::kOrderNone, order_n = 0;
  uint16_t order[mbe::kMaxOrder];
};

// Work units the chip runs at once: 256 CUs, one 256-row workgroup each.
constexpr int64_t kConcurrentUnits = 256;
constexpr int64_t kMinChunk = 128;      // shortest split, in keys
constexpr int kCusPerXcd = 32;

// Cost model of a dispatch table, in 64-key tile times: a work unit costs
// its tiles plus a workgroup's start (Q and the first tiles' latency, about
// four tile times); splitting adds the merge (its launch, and reading the
// partial results at roughly 8 MB per tile time).
constexpr double kUnitStartTiles = 4.0;
constexpr double kMergeStartTiles = 1.5;
constexpr double kMergeBytesPerTile = 8e6;
constexpr double kMinPlanGain = 0.01;   // a shorter split must beat the default by this share

struct SeqWork {
  int64_t n;      // keys the sequence's units read (0: no rows)
  int64_t w;      // window rows
  int32_t nq;     // query tiles with rows
};

struct UnitSchedule {
  double finish = -1.0;           // modelled completion in tile times; < 0: no table
  int32_t order_n = 0;            // workgroups: 8 x the longest XCD list
  uint16_t order[mbe::kMaxOrder]; // workgroup id -> work unit (kNoUnit: none)
};

// Dispatch table for splits of c keys.  The work units that have rows and
// keys form groups (the query tiles of one (split, sequence, KV head), which
// read the same keys); the groups are dealt largest first to the XCD with
// the least work so far, and an XCD's units take its slots (workgroup ids x,
// x + 8, ...) in that order, so that each XCD starts its longest units first
// and the hardware, which starts an XCD's next workgroup on whichever of its
// CUs frees first, balances them.  The modelled finish replays exactly
// that.  No table (finish < 0) with more than kMaxOrder units, more than
// kMaxOrder / 8 on one XCD, or a unit index beyond 16 bits.
void schedule_units(const std::vector<SeqWork> &seqs, int32_t hkv, int32_t qtiles, int32_t hq, int32_t head_dim,
                    int64_t max_kv, int64_t c, UnitSchedule *out) {
  out->finish = -1.0;
  const int64_t batch = static_cast<int64_t>(seqs.size());
  const int64_t splits = std::max<int64_t>(1, (max_kv + c - 1) / c);
  const int64_t per_split = batch * hkv;
  if (per_split * splits * qtiles >= mbe::kNoUnit) return;
  auto nsplit_of = [&](int64_t n) { return std::min<int64_t>(splits, std::max<int64_t>(1, (n + c - 1) / c)); };
  int64_t total = 0;
  bool same_nq = true;
  for (const SeqWork &sq : seqs)
    if (sq.n > 0) {
      total += nsplit_of(sq.n) * hkv * sq.nq;
      same_nq = same_nq && sq.nq == seqs[0].nq;
    }
  if (total == 0 || total > mbe::kMaxOrder) return;

  struct Grp {
    float cost;
    int32_t grp;
    int16_t nq, tiles;
  };
  Grp grps[mbe::kMaxOrder];
  int ng = 0;
  double merge_bytes = 0.0;
  bool any_split = false;
  auto add = [&](int64_t b, int64_t sp, int64_t keys) {
    const int t = static_cast<int>(std::min<int64_t>((keys + mbe::kKeyTile - 1) / mbe::kKeyTile, 32767));
    const int32_t nq = seqs[b].nq;
    for (int32_t g = 0; g < hkv; ++g)
      grps[ng++] = {static_cast<float>(nq * (t + kUnitStartTiles)), static_cast<int32_t>(sp * per_split + b * hkv + g),
                    static_cast<int16_t>(nq), static_cast<int16_t>(t)};
  };
  // Largest first.  With the same query tiles for every sequence this order
  // needs no sort over the groups: every full-length split (c keys) first,
  // then each sequence's last split by its length.
  struct Last {
    int64_t keys, b;
  };
  Last last[mbe::kMaxOrder];
  int nl = 0;
  for (int64_t b = 0; b < batch; ++b) {
    const SeqWork &sq = seqs[b];
    if (sq.n == 0) continue;
    const int64_t nsb = nsplit_of(sq.n);
    if (nsb > 1) {
      any_split = true;
      // partial O and (reference, sum) read per split, bf16 O written
      merge_bytes += static_cast<double>(sq.w) * hq * (nsb * (head_dim + 2) * 4.0 + head_dim * 2.0);
    }
    for (int64_t sp = 0; sp + 1 < nsb; ++sp) add(b, sp, c);
    last[nl++] = {sq.n - (nsb - 1) * c, b};
  }
  std::sort(last, last + nl, [](const Last &x, const Last &y) { return x.keys != y.keys ? x.keys > y.keys : x.b < y.b; });
  for (int i = 0; i < nl; ++i) add(last[i].b, nsplit_of(seqs[last[i].b].n) - 1, last[i].keys);
  if (!same_nq) std::stable_sort(grps, grps + ng, [](const Grp &x, const Grp &y) { return x.cost > y.cost; });

  constexpr int kSlots = mbe::kMaxOrder / mbe::kXcds;
  uint16_t unit[mbe::kXcds][kSlots];
  int16_t tiles[mbe::kXcds][kSlots];
  int len[mbe::kXcds] = {};
  double load[mbe::kXcds] = {};
  for (int i = 0; i < ng; ++i) {
    int x = 0;                     // least-loaded XCD, lowest index on ties (selects, no branches)
    double lx = load[0];
    for (int j = 1; j < mbe::kXcds; ++j) {
      const bool lt = load[j] < lx;
      x = lt ? j : x;
      lx = lt ? load[j] : lx;
    }
    if (len[x] + grps[i].nq > kSlots) return;
    load[x] += grps[i].cost;
    for (int q = 0; q < grps[i].nq; ++q) {
      unit[x][len[x]] = static_cast<uint16_t>(grps[i].grp * qtiles + q);
      tiles[x][len[x]++] = grps[i].tiles;
    }
  }
  // replay: per XCD, each unit starts on the CU that frees first: the first
  // 32 take one CU each, the rest go through a min-heap of the CU free times
  float finish = 0.f;
  for (int x = 0; x < mbe::kXcds; ++x) {
    const int first = std::min(len[x], kCusPerXcd);
    float heap[kCusPerXcd];
    float end = 0.f;
    for (int j = 0; j < first; ++j) {
      heap[j] = tiles[x][j] + static_cast<float>(kUnitStartTiles);
      end = std::max(end, heap[j]);
    }
    if (len[x] > kCusPerXcd) {
      std::make_heap(heap, heap + kCusPerXcd, std::greater<float>());
      for (int j = kCusPerXcd; j < len[x]; ++j) {
        std::pop_heap(heap, heap + kCusPerXcd, std::greater<float>());
        const float t = heap[kCusPerXcd - 1] + tiles[x][j] + static_cast<float>(kUnitStartTiles);
        heap[kCusPerXcd - 1] = t;
        std::push_heap(heap, heap + kCusPerXcd, std::greater<float>());
        end = std::max(end, t);
      }
    }
    finish = std::max(finish, end);
  }
  if (any_split) finish += static_cast<float>(kMergeStartTiles + merge_bytes / kMergeBytesPerTile);
  int slots = 0;
  for (int x = 0; x < mbe::kXcds; ++x) slots = std::max(slots, len[x]);
  out->finish = finish;
  out->order_n = slots * mbe::kXcds;
  for (int j = 0; j < slots; ++j)
    for (int x = 0; x < mbe::kXcds; ++x) out->order[j * mbe::kXcds + x] = j < len[x] ? unit[x][j] : mbe::kNoUnit;
}

mbe_status plan_attention(const mbe_paged_kv *kv, const mbe_attn_opts *o, int32_t block_size,
                          int32_t window_bound, int32_t fixed_window, AttnPlan *pl) {
  if (!kv) return fail(MBE_ERR_NULL_ARG, "paged_kv is NULL");
  if (!o) return fail(MBE_ERR_NULL_ARG, "opts is NULL");
  if (kv->page_size != mbe::kPageSize)
    return fail(MBE_ERR_UNSUPPORTED, "page_size %d: only 16-token pages are supported", kv->page_size);
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(MBE_ERR_UNSUPPORTED, "head_dim %d: supported are 64 and 128", kv->head_dim);
  if (kv->num_kv_heads < 1) return fail(MBE_ERR_BAD_SHAPE, "num_kv_heads %d < 1", kv->num_kv_heads);
  if (kv->v_layout != MBE_V_TOKEN_MINOR && kv->v_layout != MBE_V_TOKEN_MAJOR)
    return fail(MBE_ERR_UNSUPPORTED, "v_layout %d", kv->v_layout);
  if (kv->num_pages < 0) return fail(MBE_ERR_BAD_SHAPE, "num_pages %d < 0", kv->num_pages);
  if (o->batch < 0) return fail(MBE_ERR_BAD_SHAPE, "batch %d < 0", o->batch);
  if (o->num_q_heads < 1 || o->num_q_heads % kv->num_kv_heads != 0)
    return fail(MBE_ERR_BAD_SHAPE, "num_q_heads %d is not a positive multiple of num_kv_heads %d",
                o->num_q_heads, kv->num_kv_heads);
  if (block_size < 1) return fail(MBE_ERR_BAD_SHAPE, "block_size %d < 1", block_size);
  if (o->total_q < 0 || o->max_prefix_len < 0 || window_bound < 0 || o->max_pages_per_seq < 0)
    return fail(MBE_ERR_BAD_SHAPE, "negative total_q/max_prefix_len/max_window_len/max_pages_per_seq");
  if (window_bound % block_size != 0)
    return fail(MBE_ERR_BAD_SHAPE, "max_window_len %d is not a multiple of block_size %d", window_bound,
                block_size);
  if (o->mask_mode != MBE_MASK_WINDOW_BIDIR && o->mask_mode != MBE_MASK_BLOCK_CAUSAL)
    return fail(MBE_ERR_UNSUPPORTED, "mask_mode %d", o->mask_mode);
  if (o->softmax_scale != o->softmax_scale) return fail(MBE_ERR_BAD_VALUE, "softmax_scale is NaN");
  if (o->kv_split_tokens < 0 || o->kv_split_tokens % mbe::kKeyTile != 0)
    return fail(MBE_ERR_BAD_SHAPE, "kv_split_tokens %d is not 0 or a positive multiple of 64",
                o->kv_split_tokens);
  const int64_t max_kv = static_cast<int64_t>(o->max_prefix_len) + window_bound;
  if (o->batch > 0 && max_kv > 0 && o->max_pages_per_seq < 1)
    return fail(MBE_ERR_BAD_SHAPE, "max_pages_per_seq must be >= 1");
  if (max_kv > (1LL << 30)) return fail(MBE_ERR_BAD_SHAPE, "sequence bound too large");
  if (o->batch > 0 && kv->num_pages < 1 && max_kv > 0) return fail(MBE_ERR_BAD_SHAPE, "empty page pool");

  pl->group = o->num_q_heads / kv->num_kv_heads;
  const int64_t rows = static_cast<int64_t>(pl->group) * window_bound;
  pl->qtiles = static_cast<int32_t>(std::max<int64_t>(1, (rows + mbe::kRowsPerTile - 1) / mbe::kRowsPerTile));
  const int64_t base_units = static_cast<int64_t>(o->batch) * kv->num_kv_heads * pl->qtiles;

  // Host copies of the lengths, when given, refine the plan.
  const bool host = o->host_prefix_lens && (fixed_window >= 0 || o->host_window_lens) &&
                    o->batch > 0 && o->batch <= mbe::kMaxOrder;
  std::vector<int64_t> n_seq;   // keys each sequence's units read
  if (host) {
    n_seq.resize(o->batch);
    for (int b = 0; b < o->batch; ++b) {
      const int64_t P = o->host_prefix_lens[b];
      const int64_t W = fixed_window >= 0 ? fixed_window : o->host_window_lens[b];
      if (P < 0 || P > o->max_prefix_len || W < 0 || W > window_bound)
        return fail(MBE_ERR_BAD_SHAPE, "host lengths of sequence %d (%lld, %lld) exceed the bounds", b,
                    static_cast<long long>(P), static_cast<long long>(W));
      n_seq[b] = W > 0 ? P + W : 0;
    }
  }

  int64_t chunk = o->kv_split_tokens;
  bool rule_split = false;      // the default rule below cut the key ranges to fill the CUs
  if (chunk == 0) {
    // Work units (sequence, KV head, query tile, split) with splits of c keys.
    auto units = [&](int64_t c) {
      int64_t u = 0;
      if (host) {
        for (int b = 0; b < o->batch; ++b) {
          if (n_seq[b] == 0) continue;
          const int64_t W = fixed_window >= 0 ? fixed_window : o->host_window_lens[b];
          const int64_t qt = (pl->group * W + mbe::kRowsPerTile - 1) / mbe::kRowsPerTile;
          u += kv->num_kv_heads * qt * ((n_seq[b] + c - 1) / c);
        }
      } else {
        u = base_units * ((max_kv + c - 1) / c);
      }
      return u;
    };
    const int64_t c_max = std::max<int64_t>(kMinChunk, (max_kv + mbe::kKeyTile - 1) / mbe::kKeyTile * mbe::kKeyTile);
    if (units(c_max) > kConcurrentUnits) {
      // More units than CUs already: no split (each split adds a pipeline fill
      // and a merge of partial results, and the longest-first order balances
      // the units of a large batch).
      chunk = c_max;
    } else {
      // Splits as short as possible while every unit still starts in the first
      // round on the 256 CUs: the smallest multiple of 64 keys whose unit count
      // fits (the count only falls as the split grows).
      int64_t lo = std::max<int64_t>(kMinChunk / mbe::kKeyTile, 1), hi = c_max / mbe::kKeyTile;
      while (lo < hi) {
        const int64_t mid = (lo + hi) / 2;
        if (units(mid * mbe::kKeyTile) <= kConcurrentUnits) hi = mid;
        else lo = mid + 1;
      }
      chunk = lo * mbe::kKeyTile;
      rule_split = true;
    }
  }
  chunk = std::max<int64_t>(mbe::kKeyTile, (chunk + mbe::kKeyTile - 1) / mbe::kKeyTile * mbe::kKeyTile);

  // Ragged small batches (the rule above split them, and the lengths
  // differ): a dispatch table that balances the units over the XCDs and CUs,
  // for the default split length or 7/8 or 3/4 of it, whichever the model
  // finishes first (the default unless another beats it by kMinPlanGain).
  // Equal lengths are balanced by the formula already, and large batches
  // gained nothing from a table.
  UnitSchedule sched;
  if (host && rule_split) {
    bool ragged = false;
    for (int b = 1; b < o->batch; ++b) ragged = ragged || n_seq[b] != n_seq[0];
    if (ragged) {
      std::vector<SeqWork> seqs(o->batch);
      for (int b = 0; b < o->batch; ++b) {
        const int64_t W = fixed_window >= 0 ? fixed_window : o->host_window_lens[b];
        seqs[b] = {n_seq[b], W, static_cast<int32_t>((pl->group * W + mbe::kRowsPerTile - 1) / mbe::kRowsPerTile)};
      }
      schedule_units(seqs, kv->num_kv_heads, pl->qtiles, o->num_q_heads, kv->head_dim, max_kv, chunk, &sched);
      UnitSchedule alt;
      const int64_t d = chunk;
      for (int64_t cand : {d * 7 / 8, d * 3 / 4}) {
        const int64_t c = std::max<int64_t>(kMinChunk, (cand + mbe::kKeyTile - 1) / mbe::kKeyTile * mbe::kKeyTile);
        if (c >= d) continue;
        schedule_units(seqs, kv->num_kv_heads, pl->qtiles, o->num_q_heads, kv->head_dim, max_kv, c, &alt);
        if (alt.finish >= 0 && (sched.finish < 0 || alt.finish < sched.finish * (1.0 - kMinPlanGain))) {
          chunk = c;
          sched = alt;
        }
      }
    }
  }

  pl->kv_chunk = static_cast<int32_t>(std::min<int64_t>(chunk, 1LL << 30));
  pl->splits = static_cast<int32_t>(std::max<int64_t>(1, (max_kv + chunk - 1) / chunk));
  pl->groups = static_cast<int64_t>(o->batch) * kv->num_kv_heads * pl->splits;
  pl->slots_per_xcd = (pl->groups + mbe::kXcds - 1) / mbe::kXcds * pl->qtiles;
  if (pl->slots_per_xcd * mbe::kXcds > 0x7fffffffLL) return fail(MBE_ERR_BAD_SHAPE, "grid too large");

  pl->order_kind = mbe::kOrderNone;
  pl->order_n = 0;
  if (sched.finish >= 0) {
    pl->order_kind = mbe::kOrderUnits;
    pl->order_n = sched.order_n;
    std::copy(sched.order, sched.order + sched.order_n, pl->order);
  } else if (host) {
    // Longest sequences first (stable), so the short ones fill in at the end
    // (no table when that is the natural order, e.g. one sequence or equal
    // lengths: the kernel then skips reading it).
    std::vector<int32_t> idx(o->batch);
    for (int b = 0; b < o->batch; ++b) idx[b] = b;
    std::stable_sort(idx.begin(), idx.end(), [&](int32_t x, int32_t y) { return n_seq[x] > n_seq[y]; });
    bool natural = true;
    for (int b = 0; b < o->batch; ++b) {
      pl->order[b] = static_cast<uint16_t>(idx[b]);
      natural = natural && idx[b] == b;
    }
    if (!natural) {
      pl->order_kind = mbe::kOrderSeqs;
      pl->order_n = o->batch;
    }
  }

  pl->bytes = 0;
  if (pl->splits > 1) {
    const size_t rows_all = static_cast<size_t>(pl->splits) * o->total_q * o->num_q_heads;
    pl->part_o_off = 0;
    pl->part_ml_off = align_up(rows_all * kv->head_dim * sizeof(float));
    pl->bytes = pl->part_ml_off + align_up(rows_all * 2 * sizeof(float));
  }
  return MBE_OK;
}

mbe_status debug_check_attention(const mbe_paged_kv *kv, const int32_t *page_table, const int32_t *prefix_lens,
                                 const int32_t *window_lens, int32_t block_size, int32_t fixed_window,
                                 const mbe_attn_opts *o) {
  const int B = o->batch;
  const hipStream_t stream = static_cast<hipStream_t>(o->stream);
  // A copy cannot be recorded into a graph: calls made while the stream is
  // capturing are not checked.
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e != hipSuccess) return hip_fail(e, "MBE_DEBUG_CHECK capture query");
  if (cs != hipStreamCaptureStatusNone) return MBE_OK;
  // copies on the call's stream, so they see what the caller wrote there before
  std::vector<int32_t> P(B), W(B, fixed_window), T(static_cast<size_t>(B) * o->max_pages_per_seq);
  e = hipMemcpyAsync(P.data(), prefix_lens, B * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess && fixed_window < 0)
    e = hipMemcpyAsync(W.data(), window_lens, B * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess && !T.empty())
    e = hipMemcpyAsync(T.data(), page_table, T.size() * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "MBE_DEBUG_CHECK copy");
  int64_t tq = 0;
  for (int b = 0; b < B; ++b) {
    if (P[b] < 0 || P[b] > o->max_prefix_len)
      return fail(MBE_ERR_BAD_VALUE, "prefix_lens[%d] = %d outside [0, %d]", b, P[b], o->max_prefix_len);
    const int wb = fixed_window >= 0 ? fixed_window : o->max_window_len;
    if (W[b] < 0 || W[b] > wb || W[b] % block_size != 0)
      return fail(MBE_ERR_BAD_VALUE, "window_lens[%d] = %d invalid", b, W[b]);
    tq += W[b];
    const int np = (P[b] + W[b] + mbe::kPageSize - 1) / mbe::kPageSize;
    if (np > o->max_pages_per_seq)
      return fail(MBE_ERR_BAD_VALUE, "sequence %d needs %d pages > max_pages_per_seq %d", b, np,
                  o->max_pages_per_seq);
    for (int j = 0; j < np; ++j) {
      const int32_t pg = T[static_cast<size_t>(b) * o->max_pages_per_seq + j];
      if (pg < 0 || pg >= kv->num_pages)
        return fail(MBE_ERR_BAD_VALUE, "page_table[%d][%d] = %d outside [0, %d)", b, j, pg, kv->num_pages);
    }
  }
  if (tq != o->total_q)
    return fail(MBE_ERR_BAD_VALUE, "sum of window lengths %lld != total_q %d", static_cast<long long>(tq),
                o->total_q);
  return MBE_OK;
}

// MBE_DEBUG_CHECK for the KV write-back: every written position must lie in
// its sequence's table row and its page id in the pool, and the lengths must
// fit the bounds and the rows of the input.
mbe_status debug_check_kv_write(const int32_t *page_table, int32_t max_pages, int32_t num_pages,
                                const int32_t *start_pos, const int32_t *lens, int32_t batch, int32_t max_len,
                                int32_t total_tokens, hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e != hipSuccess) return hip_fail(e, "MBE_DEBUG_CHECK capture query");
  if (cs != hipStreamCaptureStatusNone) return MBE_OK;
  std::vector<int32_t> S(batch), L(batch), T(static_cast<size_t>(batch) * max_pages);
  e = hipMemcpyAsync(S.data(), start_pos, batch * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(L.data(), lens, batch * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(T.data(), page_table, T.size() * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "MBE_DEBUG_CHECK copy");
  int64_t rows = 0;
  for (int b = 0; b < batch; ++b) {
    if (L[b] < 0 || L[b] > max_len) return fail(MBE_ERR_BAD_VALUE, "lens[%d] = %d outside [0, %d]", b, L[b], max_len);
    if (S[b] < 0) return fail(MBE_ERR_BAD_VALUE, "start_pos[%d] = %d < 0", b, S[b]);
    rows += L[b];
    if (L[b] == 0) continue;
    const int64_t last = (static_cast<int64_t>(S[b]) + L[b] - 1) / mbe::kPageSize;
    if (last >= max_pages)
      return fail(MBE_ERR_BAD_VALUE, "sequence %d writes up to position %lld, past its %d table pages", b,
                  static_cast<long long>(S[b]) + L[b] - 1, max_pages);
    for (int64_t j = S[b] / mbe::kPageSize; j <= last; ++j) {
      const int32_t pg = T[static_cast<size_t>(b) * max_pages + j];
      if (pg < 0 || pg >= num_pages)
        return fail(MBE_ERR_BAD_VALUE, "page_table[%d][%lld] = %d outside [0, %d)", b, static_cast<long long>(j), pg,
                    num_pages);
    }
  }
  if (rows != total_tokens)
    return fail(MBE_ERR_BAD_VALUE, "sum of lens %lld != total_tokens %d", static_cast<long long>(rows), total_tokens);
  return MBE_OK;
}

// At most 128 rows per (sequence, KV head): two waves per 32 rows, each
// taking half of every key tile, instead of four waves with no rows.
int32_t key_split_of(const AttnPlan &pl, int32_t window_bound) {
  return static_cast<int64_t>(pl.group) * window_bound <= mbe::kRowsPerTile / 2 ? 2 : 1;
}

bool use_pipelined(const mbe_paged_kv *kv, const mbe_attn_opts *o, const AttnPlan &pl, int32_t window_bound,
                   int32_t key_split) {
  const int64_t unit_keys = std::min<int64_t>(pl.kv_chunk, static_cast<int64_t>(o->max_prefix_len) + window_bound);
  const int force = pipeline_override();
  const bool eligible = kv->v_layout != MBE_V_TOKEN_MAJOR && key_split == 1;
  return eligible && (force >= 0 ? force == 1 : (unit_keys + mbe::kKeyTile - 1) / mbe::kKeyTile >= kPipeMinTiles);
}

mbe_status run_attention(const void *q, const mbe_paged_kv *kv, const int32_t *page_table,
                         const int32_t *prefix_lens, const int32_t *window_lens, int32_t block_size,
                         int32_t fixed_window, void *out, const mbe_attn_opts *o) {
  const int32_t window_bound = fixed_window >= 0 ? fixed_window : (o ? o->max_window_len : 0);
  AttnPlan pl;
  mbe_status st = plan_attention(kv, o, block_size, window_bound, fixed_window, &pl);
  if (st != MBE_OK) return st;
  if (fixed_window >= 0 && o->total_q != static_cast<int64_t>(o->batch) * fixed_window)
    return fail(MBE_ERR_BAD_SHAPE, "total_q %d != batch %d * block_size %d", o->total_q, o->batch,
                fixed_window);
  if (o->batch == 0 || o->total_q == 0) return MBE_OK;
  if (!q || !out || !page_table || !prefix_lens || !kv->k_pages || !kv->v_pages)
    return fail(MBE_ERR_NULL_ARG, "q, out, page_table, prefix_lens, k_pages and v_pages must be non-NULL");
  if (fixed_window < 0 && !window_lens) return fail(MBE_ERR_NULL_ARG, "window_lens is NULL");
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(out) |
       reinterpret_cast<uintptr_t>(kv->k_pages) | reinterpret_cast<uintptr_t>(kv->v_pages)) % 16 != 0)
    return fail(MBE_ERR_BAD_SHAPE, "q, out, k_pages and v_pages must be 16-byte aligned");
  if (pl.bytes > 0) {
    if (!o->workspace) return fail(MBE_ERR_WORKSPACE, "workspace of %zu bytes required", pl.bytes);
    if (o->workspace_bytes < pl.bytes)
      return fail(MBE_ERR_WORKSPACE, "workspace %zu bytes < required %zu", o->workspace_bytes, pl.bytes);
    if (reinterpret_cast<uintptr_t>(o->workspace) % 256 != 0)
      return fail(MBE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }
  if (debug_checks()) {
    st = debug_check_attention(kv, page_table, prefix_lens, window_lens, block_size, fixed_window, o);
    if (st != MBE_OK) return st;
  }

  mbe::AttnParams p{};
  p.q = static_cast<const uint16_t *>(q);
  p.k_pages = static_cast<const uint16_t *>(kv->k_pages);
  p.v_pages = static_cast<const uint16_t *>(kv->v_pages);
  p.page_table = page_table;
  p.prefix_lens = prefix_lens;
  p.window_lens = window_lens;
  p.out = static_cast<uint16_t *>(out);
  char *ws = static_cast<char *>(o->workspace);
  p.part_o = pl.bytes ? reinterpret_cast<float *>(ws + pl.part_o_off) : nullptr;
  p.part_ml = pl.bytes ? reinterpret_cast<float *>(ws + pl.part_ml_off) : nullptr;
  p.batch = o->batch;
  p.num_q_heads = o->num_q_heads;
  p.num_kv_heads = kv->num_kv_heads;
  p.group = pl.group;
  p.num_pages = kv->num_pages;
  p.max_pages = o->max_pages_per_seq;
  p.block_size = block_size;
  p.total_q = o->total_q;
  p.fixed_window = fixed_window;
  p.max_prefix = o->max_prefix_len;
  p.max_window = window_bound;
  p.qtiles = pl.qtiles;
  p.key_split = key_split_of(pl, window_bound);
  p.v_token_major = kv->v_layout == MBE_V_TOKEN_MAJOR;
  p.pipelined = use_pipelined(kv, o, pl, window_bound, p.key_split);
  p.splits = pl.splits;
  p.kv_chunk = pl.kv_chunk;
  p.groups = pl.groups;
  p.slots_per_xcd = pl.slots_per_xcd;
  p.order_kind = pl.order_kind;
  p.order_n = pl.order_n;
  for (int i = 0; i < pl.order_n; ++i) p.order[i] = pl.order[i];
  const float scale = o->softmax_scale > 0.f ? o->softmax_scale : 1.0f / std::sqrt(static_cast<float>(kv->head_dim));
  p.scale_log2 = scale * 1.4426950408889634f;
  p.block_flags = o->block_flags;
  p.flag_stride = window_bound / block_size;
  p.gate = o->run_if_nonzero;
  const int mode = fixed_window >= 0 ? MBE_MASK_WINDOW_BIDIR : o->mask_mode;
  hipError_t e = mbe::launch_window_attention(p, kv->head_dim, mode, static_cast<hipStream_t>(o->stream));
  if (e != hipSuccess) return hip_fail(e, "window attention launch");
  return MBE_OK;
}

}  // namespace

namespace mbe {

void edit_select_plan(int64_t rows, int64_t vocab, int32_t *chunks, int64_t *chunk_len) {
  // Enough workgroups to cover the 256 CUs twice; a chunk keeps at least 4096
  // elements, one full iteration of the workgroup.  (Measured on 64 rows of
  // 131072: 512 workgroups of 4 iterations beat 2048 of one, whose time is
  // dispatch and one memory round trip.)
  const int64_t target_wgs = 512;
  int64_t c = 1;
  if (rows < target_wgs) {
    c = (target_wgs + rows - 1) / rows;
    const int64_t max_c = (vocab + 4095) / 4096;
    if (c > max_c) c = max_c;
    if (c > 1024) c = 1024;
    if (c < 1) c = 1;
  }
  int64_t len = (vocab + c - 1) / c;
  len = (len + 7) / 8 * 8;
  c = (vocab + len - 1) / len;
  if (c < 1) c = 1;
  *chunks = static_cast<int32_t>(c);
  *chunk_len = len;
}

mbe_status report(mbe_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

mbe_status threshold_update_check(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                  const int32_t *cur_tokens, int32_t block_size, float omega_mask, float omega_edit,
                                  const int32_t *new_tokens, const float *conf, const uint8_t *action,
                                  const uint8_t *block_changed, const int32_t *changed_count,
                                  const int32_t *run_if_nonzero, size_t *need) {
  *need = 0;
  if (rows < 0 || vocab < 0) return fail(MBE_ERR_BAD_SHAPE, "rows %lld / vocab %lld negative",
                                         static_cast<long long>(rows), static_cast<long long>(vocab));
  if (rows > 0 && vocab < 1) return fail(MBE_ERR_BAD_SHAPE, "vocab must be >= 1");
  if (row_stride < vocab)
    return fail(MBE_ERR_BAD_SHAPE, "row_stride %lld < vocab %lld", static_cast<long long>(row_stride),
                static_cast<long long>(vocab));
  if (vocab > 0x7fffffffLL) return fail(MBE_ERR_BAD_SHAPE, "vocab beyond int32 indices");
  if (block_size < 1) return fail(MBE_ERR_BAD_SHAPE, "block_size %d < 1", block_size);
  if (rows % block_size != 0)
    return fail(MBE_ERR_BAD_SHAPE, "rows %lld is not a multiple of block_size %d", static_cast<long long>(rows),
                block_size);
  if (omega_mask != omega_mask || omega_edit != omega_edit) return fail(MBE_ERR_BAD_VALUE, "threshold is NaN");
  if (run_if_nonzero && run_if_nonzero == changed_count)
    return fail(MBE_ERR_BAD_VALUE, "run_if_nonzero must not be changed_count itself (the pass zeroes it)");
  if (rows == 0) return MBE_OK;
  if (!logits || !cur_tokens || !new_tokens || !conf || !action || !block_changed)
    return fail(MBE_ERR_NULL_ARG, "logits, cur_tokens, new_tokens, conf, action and block_changed must be non-NULL");
  int32_t chunks;
  int64_t len;
  edit_select_plan(rows, vocab, &chunks, &len);
  if (rows * chunks > 0x7fffffffLL) return fail(MBE_ERR_BAD_SHAPE, "too many rows");
  *need = mbe_threshold_update_workspace_size(rows, vocab);
  return MBE_OK;
}

mbe_status threshold_update_launch(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                   const int32_t *cur_tokens, int32_t mask_id, int32_t block_size, float omega_mask,
                                   float omega_edit, int32_t *new_tokens, float *conf, uint8_t *action,
                                   uint8_t *block_changed, int32_t *changed_count, float *entropy,
                                   const int32_t *run_if_nonzero, void *workspace, void *stream) {
  int32_t chunks;
  int64_t len;
  edit_select_plan(rows, vocab, &chunks, &len);
  EsParams p{};
  p.logits = static_cast<const uint16_t *>(logits);
  p.rows = rows;
  p.vocab = vocab;
  p.ld = row_stride;
  p.chunk_len = len;
  p.chunks = chunks;
  p.update = 1;
  p.cur = cur_tokens;
  p.threshold = omega_edit;
  p.new_tokens = new_tokens;
  p.conf = conf;
  char *ws = static_cast<char *>(workspace);
  p.pred = reinterpret_cast<int32_t *>(ws);
  if (chunks > 1) p.partials = reinterpret_cast<EsPartial *>(ws + align_up(static_cast<size_t>(rows) * 4));
  p.entropy = entropy;
  p.changed_count = changed_count;
  p.action = action;
  p.block_changed = block_changed;
  p.mask_id = mask_id;
  p.block_size = block_size;
  p.omega_mask = omega_mask;
  p.gate = run_if_nonzero;
  const bool vec = (reinterpret_cast<uintptr_t>(logits) % 16 == 0) && (row_stride % 8 == 0);
  hipError_t e = launch_threshold_update(p, vec, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "threshold update launch");
  return MBE_OK;
}

}  // namespace mbe

extern "C" {

mbe_status mbe_window_attention(const void *q, const mbe_paged_kv *paged_kv, const int32_t *page_table,
                                const int32_t *prefix_lens, const int32_t *window_lens, int32_t block_size,
                                void *out, const mbe_attn_opts *opts) {
  return run_attention(q, paged_kv, page_table, prefix_lens, window_lens, block_size, -1, out, opts);
}

mbe_status block_diffusion_attention(const void *q, const mbe_paged_kv *paged_kv, const int32_t *page_table,
                                     const int32_t *prefix_lens, int32_t block_size, void *out,
                                     const mbe_attn_opts *opts) {
  if (block_size < 1) return fail(MBE_ERR_BAD_SHAPE, "block_size %d < 1", block_size);
  return run_attention(q, paged_kv, page_table, prefix_lens, nullptr, block_size, block_size, out, opts);
}

mbe_status mbe_window_attention_plan(const mbe_paged_kv *paged_kv, const mbe_attn_opts *opts, mbe_attn_plan *plan) {
  if (!opts || !plan) return fail(MBE_ERR_NULL_ARG, "opts and plan must not be NULL");
  AttnPlan pl;
  const mbe_status st = plan_attention(paged_kv, opts, 1, opts->max_window_len, -1, &pl);
  if (st != MBE_OK) return st;
  const int32_t ks = key_split_of(pl, opts->max_window_len);
  plan->splits = pl.splits;
  plan->kv_chunk = pl.kv_chunk;
  plan->key_split = ks;
  plan->pipelined = use_pipelined(paged_kv, opts, pl, opts->max_window_len, ks) ? 1 : 0;
  plan->workgroups = pl.order_kind == mbe::kOrderUnits ? pl.order_n : pl.slots_per_xcd * mbe::kXcds;
  return MBE_OK;
}

size_t mbe_window_attention_workspace_size(const mbe_paged_kv *paged_kv, const mbe_attn_opts *opts) {
  // The split plan of a window call does not depend on the block size (only
  // the call's check that the window bound is a multiple of it does), so the
  // plan is made with block size 1.
  AttnPlan pl;
  if (!opts) return static_cast<size_t>(-1);
  if (plan_attention(paged_kv, opts, 1, opts->max_window_len, -1, &pl) != MBE_OK)
    return static_cast<size_t>(-1);
  return pl.bytes;
}

size_t mbe_block_diffusion_workspace_size(const mbe_paged_kv *paged_kv, const mbe_attn_opts *opts,
                                          int32_t block_size) {
  AttnPlan pl;
  if (!opts || block_size < 1) return static_cast<size_t>(-1);
  if (plan_attention(paged_kv, opts, block_size, block_size, block_size, &pl) != MBE_OK)
    return static_cast<size_t>(-1);
  return pl.bytes;
}

size_t mbe_edit_select_workspace_size(int64_t rows, int64_t vocab) {
  if (rows < 0 || vocab < 0) return static_cast<size_t>(-1);
  if (rows == 0 || vocab == 0) return 0;
  int32_t chunks;
  int64_t len;
  mbe::edit_select_plan(rows, vocab, &chunks, &len);
  if (chunks <= 1) return 0;
  return align_up(static_cast<size_t>(rows) * chunks * sizeof(mbe::EsPartial));
}

mbe_status mbe_edit_select(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                           const int32_t *cur_tokens, float threshold, int32_t *new_tokens, float *conf,
                           uint8_t *changed_mask, void *workspace, size_t workspace_bytes, void *stream) {
  if (rows < 0 || vocab < 0) return fail(MBE_ERR_BAD_SHAPE, "rows %lld / vocab %lld negative",
                                         static_cast<long long>(rows), static_cast<long long>(vocab));
  if (rows > 0 && vocab < 1) return fail(MBE_ERR_BAD_SHAPE, "vocab must be >= 1");
  if (row_stride < vocab)
    return fail(MBE_ERR_BAD_SHAPE, "row_stride %lld < vocab %lld", static_cast<long long>(row_stride),
                static_cast<long long>(vocab));
  if (vocab > 0x7fffffffLL) return fail(MBE_ERR_BAD_SHAPE, "vocab beyond int32 indices");
  if (threshold != threshold) return fail(MBE_ERR_BAD_VALUE, "threshold is NaN");
  if (rows == 0) return MBE_OK;
  if (!logits || !cur_tokens || !new_tokens || !conf || !changed_mask)
    return fail(MBE_ERR_NULL_ARG, "logits, cur_tokens, new_tokens, conf and changed_mask must be non-NULL");
  int32_t chunks;
  int64_t len;
  mbe::edit_select_plan(rows, vocab, &chunks, &len);
  if (rows * chunks > 0x7fffffffLL) return fail(MBE_ERR_BAD_SHAPE, "too many rows");
  const size_t need = mbe_edit_select_workspace_size(rows, vocab);
  if (need > 0) {
    if (!workspace) return fail(MBE_ERR_WORKSPACE, "workspace of %zu bytes required", need);
    if (workspace_bytes < need)
      return fail(MBE_ERR_WORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
      return fail(MBE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }
  mbe::EsParams p{};
  p.logits = static_cast<const uint16_t *>(logits);
  p.rows = rows;
  p.vocab = vocab;
  p.ld = row_stride;
  p.chunk_len = len;
  p.chunks = chunks;
  p.cur = cur_tokens;
  p.threshold = threshold;
  p.new_tokens = new_tokens;
  p.conf = conf;
  p.changed = changed_mask;
  if (need > 0) {
    char *ws = static_cast<char *>(workspace);
    p.partials = reinterpret_cast<mbe::EsPartial *>(ws);
  }
  const bool vec = (reinterpret_cast<uintptr_t>(logits) % 16 == 0) && (row_stride % 8 == 0);
  hipError_t e = mbe::launch_edit_select(p, vec, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "edit select launch");
  return MBE_OK;
}

size_t mbe_threshold_update_workspace_size(int64_t rows, int64_t vocab) {
  if (rows < 0 || vocab < 0) return static_cast<size_t>(-1);
  if (rows == 0) return 0;
  const size_t partials = mbe_edit_select_workspace_size(rows, vocab);
  return align_up(static_cast<size_t>(rows) * sizeof(int32_t)) + partials;   // predictions, then partials
}

mbe_status mbe_threshold_update(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                const int32_t *cur_tokens, int32_t mask_id, int32_t block_size, float omega_mask,
                                float omega_edit, int32_t *new_tokens, float *conf, uint8_t *action,
                                uint8_t *block_changed, int32_t *changed_count, float *entropy,
                                const int32_t *run_if_nonzero, void *workspace, size_t workspace_bytes,
                                void *stream) {
  size_t need = 0;
  mbe_status st = mbe::threshold_update_check(logits, rows, vocab, row_stride, cur_tokens, block_size, omega_mask,
                                              omega_edit, new_tokens, conf, action, block_changed, changed_count,
                                              run_if_nonzero, &need);
  if (st != MBE_OK || rows == 0) return st;
  if (!workspace) return fail(MBE_ERR_WORKSPACE, "workspace of %zu bytes required", need);
  if (workspace_bytes < need)
    return fail(MBE_ERR_WORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(MBE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return mbe::threshold_update_launch(logits, rows, vocab, row_stride, cur_tokens, mask_id, block_size, omega_mask,
                                      omega_edit, new_tokens, conf, action, block_changed, changed_count, entropy,
                                      run_if_nonzero, workspace, stream);
}

mbe_status mbe_tail_entropy_scores(const float *entropy, int64_t num_blocks, int32_t block_size, float rho,
                                   float *scores, void *stream) {
  if (num_blocks < 0) return fail(MBE_ERR_BAD_SHAPE, "num_blocks %lld < 0", static_cast<long long>(num_blocks));
  if (block_size < 1 || block_size > 1024)
    return fail(MBE_ERR_UNSUPPORTED, "block_size %d outside [1, 1024]", block_size);
  if (!(rho > 0.f) || rho > 1.f) return fail(MBE_ERR_BAD_VALUE, "rho %g outside (0, 1]", static_cast<double>(rho));
  // k = ceil(rho * B), computed in double from the fp32 rho
  const double kd = std::ceil(static_cast<double>(rho) * block_size);
  const int32_t k = static_cast<int32_t>(kd);
  if (k < 1 || k > block_size) return fail(MBE_ERR_BAD_VALUE, "ceil(rho * block_size) = %d", k);
  if (num_blocks > 0x7fffffffLL) return fail(MBE_ERR_BAD_SHAPE, "too many blocks");
  if (num_blocks == 0) return MBE_OK;
  if (!entropy || !scores) return fail(MBE_ERR_NULL_ARG, "entropy and scores must be non-NULL");
  hipError_t e = mbe::launch_tail_entropy_scores(entropy, num_blocks, block_size, k, scores,
                                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "tail entropy launch");
  return MBE_OK;
}

mbe_status mbe_select_start_block(const float *scores, int32_t batch, int32_t score_stride,
                                  const int32_t *current_block, int32_t k_max, int32_t *start_block, void *stream) {
  if (batch < 0) return fail(MBE_ERR_BAD_SHAPE, "batch %d < 0", batch);
  if (score_stride < 0) return fail(MBE_ERR_BAD_SHAPE, "score_stride %d < 0", score_stride);
  if (k_max < 1) return fail(MBE_ERR_BAD_SHAPE, "k_max %d < 1", k_max);
  if (batch == 0) return MBE_OK;
  if (!current_block || !start_block || (score_stride > 0 && !scores))
    return fail(MBE_ERR_NULL_ARG, "scores, current_block and start_block must be non-NULL");
  hipError_t e = mbe::launch_select_start_block(scores, batch, score_stride, current_block, k_max, start_block,
                                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "start block launch");
  return MBE_OK;
}

mbe_status mbe_kv_write(void *k_pages, void *v_pages, int32_t num_pages, int32_t num_kv_heads, int32_t head_dim,
                        int32_t v_layout, const int32_t *page_table, int32_t max_pages_per_seq, const int32_t *start_pos,
                        const int32_t *lens, int32_t batch, int32_t max_len, int32_t total_tokens, const void *k_new,
                        const void *v_new, const uint8_t *block_flags, int32_t block_size, void *stream) {
  if (head_dim != 64 && head_dim != 128)
    return fail(MBE_ERR_UNSUPPORTED, "head_dim %d: supported are 64 and 128", head_dim);
  if (num_kv_heads < 1 || num_kv_heads > 65535) return fail(MBE_ERR_BAD_SHAPE, "num_kv_heads %d", num_kv_heads);
  if (v_layout != MBE_V_TOKEN_MINOR && v_layout != MBE_V_TOKEN_MAJOR)
    return fail(MBE_ERR_UNSUPPORTED, "v_layout %d", v_layout);
  if (batch < 0 || batch > 65535) return fail(MBE_ERR_BAD_SHAPE, "batch %d outside [0, 65535]", batch);
  if (max_len < 0 || total_tokens < 0 || num_pages < 0 || max_pages_per_seq < 0)
    return fail(MBE_ERR_BAD_SHAPE, "negative max_len/total_tokens/num_pages/max_pages_per_seq");
  if (block_flags && block_size < 1) return fail(MBE_ERR_BAD_SHAPE, "block_size %d < 1 with block flags", block_size);
  if (batch == 0 || max_len == 0 || total_tokens == 0) return MBE_OK;
  if (num_pages < 1 || max_pages_per_seq < 1) return fail(MBE_ERR_BAD_SHAPE, "empty page pool or table");
  if (!k_pages || !v_pages || !page_table || !start_pos || !lens || !k_new || !v_new)
    return fail(MBE_ERR_NULL_ARG, "pools, page_table, start_pos, lens, k_new and v_new must be non-NULL");
  if ((reinterpret_cast<uintptr_t>(k_pages) | reinterpret_cast<uintptr_t>(v_pages) |
       reinterpret_cast<uintptr_t>(k_new) | reinterpret_cast<uintptr_t>(v_new)) % 16 != 0)
    return fail(MBE_ERR_BAD_SHAPE, "pools and k_new/v_new must be 16-byte aligned");
  const int32_t flag_stride = block_flags ? (max_len + block_size - 1) / block_size : 0;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (debug_checks()) {
    mbe_status s = debug_check_kv_write(page_table, max_pages_per_seq, num_pages, start_pos, lens, batch, max_len,
                                        total_tokens, st);
    if (s != MBE_OK) return s;
  }
  mbe::KvWriteParams p{};
  p.k_pages = static_cast<uint16_t *>(k_pages);
  p.v_pages = static_cast<uint16_t *>(v_pages);
  p.num_pages = num_pages;
  p.num_kv_heads = num_kv_heads;
  p.head_dim = head_dim;
  p.v_token_major = v_layout == MBE_V_TOKEN_MAJOR;
  p.page_table = page_table;
  p.max_pages = max_pages_per_seq;
  p.start_pos = start_pos;
  p.lens = lens;
  p.batch = batch;
  p.max_len = max_len;
  p.total_tokens = total_tokens;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.block_flags = block_flags;
  p.block_size = block_flags ? block_size : 1;
  p.flag_stride = flag_stride;
  hipError_t e = mbe::launch_kv_write(p, st);
  if (e != hipSuccess) return hip_fail(e, "kv write launch");
  return MBE_OK;
}

mbe_status mbe_refresh_blocks(const uint8_t *block_changed, int32_t batch, int32_t num_blocks, int32_t mode,
                              uint8_t *refresh, void *stream) {
  if (batch < 0 || num_blocks < 0) return fail(MBE_ERR_BAD_SHAPE, "batch %d / num_blocks %d negative", batch,
                                               num_blocks);
  if (mode != MBE_REFRESH_CHANGED && mode != MBE_REFRESH_CHANGED_AND_LATER)
    return fail(MBE_ERR_UNSUPPORTED, "refresh mode %d", mode);
  if (batch == 0 || num_blocks == 0) return MBE_OK;
  if (!block_changed || !refresh) return fail(MBE_ERR_NULL_ARG, "block_changed and refresh must be non-NULL");
  hipError_t e = mbe::launch_refresh_blocks(block_changed, batch, num_blocks, mode, refresh,
                                            static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "refresh launch");
  return MBE_OK;
}

const char *mbe_status_string(mbe_status s) {
  switch (s) {
    case MBE_OK: return "ok";
    case MBE_ERR_NULL_ARG: return "null argument";
    case MBE_ERR_BAD_SHAPE: return "bad shape";
    case MBE_ERR_UNSUPPORTED: return "unsupported";
    case MBE_ERR_WORKSPACE: return "workspace missing or too small";
    case MBE_ERR_HIP: return "HIP error";
    case MBE_ERR_BAD_VALUE: return "bad value";
  }
  return "unknown status";
}

const char *mbe_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
