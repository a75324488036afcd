// Host-only stand-ins for the kernel launchers of libmbe, so that the C ABI
// (abi.cpp: validation, split planning, dispatch tables, workspace sizing) can
// be built with a host compiler and run under AddressSanitizer and
// UndefinedBehaviorSanitizer without a GPU.  The attention launcher checks
// the plan it receives instead of launching: every work unit inside the grid,
// no unit twice, every unit with work present, and the split-KV partial
// results inside the workspace the caller was told to provide.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

#include "internal.h"

namespace fuzz {
// set by the driver before each call: the host lengths (or null) and the
// workspace bytes the size query returned
const int32_t *host_P = nullptr;
const int32_t *host_W = nullptr;
size_t ws_bytes = 0;
long launches = 0;
long unit_tables = 0;
}  // namespace fuzz

#define REQUIRE(c)                                                              \
  do {                                                                          \
    if (!(c)) {                                                                 \
      std::fprintf(stderr, "plan check failed: %s (line %d)\n", #c, __LINE__); \
      std::abort();                                                             \
    }                                                                           \
  } while (0)

namespace mbe {

hipError_t launch_window_attention(const AttnParams &p, int head_dim, int mask_mode, hipStream_t) {
  ++fuzz::launches;
  REQUIRE(head_dim == 64 || head_dim == 128);
  REQUIRE(mask_mode == 0 || mask_mode == 1);
  REQUIRE(p.splits >= 1 && p.kv_chunk >= kKeyTile && p.kv_chunk % kKeyTile == 0);
  REQUIRE(static_cast<int64_t>(p.splits) * p.kv_chunk >= static_cast<int64_t>(p.max_prefix) + p.max_window);
  REQUIRE(p.groups == static_cast<int64_t>(p.batch) * p.num_kv_heads * p.splits);
  REQUIRE(p.key_split == 1 || p.key_split == 2);
  // split-KV partials: [splits][total_q][Hq][D] fp32, then [splits][total_q][Hq][2]
  if (p.splits > 1) {
    const char *base = reinterpret_cast<const char *>(p.part_o);
    REQUIRE(base != nullptr && p.part_ml != nullptr);
    const size_t rows = static_cast<size_t>(p.splits) * p.total_q * p.num_q_heads;
    const char *o_end = base + rows * head_dim * sizeof(float);
    const char *ml = reinterpret_cast<const char *>(p.part_ml);
    REQUIRE(ml >= o_end);
    REQUIRE(static_cast<size_t>(ml + rows * 2 * sizeof(float) - base) <= fuzz::ws_bytes);
  }
  // the work units the kernel will find (same rules as the kernel's early exits)
  const int64_t units = p.groups * p.qtiles;
  std::vector<int> seen(static_cast<size_t>(units), 0);
  if (p.order_kind == kOrderUnits) {
    ++fuzz::unit_tables;
    REQUIRE(p.order_n > 0 && p.order_n <= kMaxOrder && p.order_n % kXcds == 0);
    for (int i = 0; i < p.order_n; ++i) {
      if (p.order[i] == kNoUnit) continue;
      REQUIRE(p.order[i] < units);
      REQUIRE(seen[p.order[i]]++ == 0);
    }
  } else {
    REQUIRE(p.slots_per_xcd * kXcds >= p.groups * p.qtiles);
    if (p.order_kind == kOrderSeqs) {
      REQUIRE(p.order_n == p.batch);
      std::vector<int> hit(p.batch, 0);
      for (int r = 0; r < p.batch; ++r) {
        REQUIRE(p.order[r] < p.batch);
        REQUIRE(hit[p.order[r]]++ == 0);
      }
    }
    for (int64_t id = 0; id < p.slots_per_xcd * kXcds; ++id) {
      const int64_t slot = id / kXcds;
      const int64_t grp = (slot / p.qtiles) * kXcds + id % kXcds;
      if (grp >= p.groups) continue;
      const int64_t u = grp * p.qtiles + slot % p.qtiles;
      REQUIRE(seen[u]++ == 0);
    }
  }
  // every unit that has rows and keys is run (when the lengths are known)
  if (fuzz::host_P && (fuzz::host_W || p.fixed_window >= 0)) {
    const int64_t per_split = static_cast<int64_t>(p.batch) * p.num_kv_heads;
    for (int64_t u = 0; u < units; ++u) {
      const int64_t grp = u / p.qtiles;
      const int qtile = static_cast<int>(u % p.qtiles);
      const int split = static_cast<int>(grp / per_split);
      const int rank = static_cast<int>((grp % per_split) / p.num_kv_heads);
      const int b = (p.order_kind == kOrderSeqs && rank < p.order_n) ? p.order[rank] : rank;
      const int W = p.fixed_window >= 0 ? p.fixed_window : fuzz::host_W[b];
      const int64_t n_all = static_cast<int64_t>(fuzz::host_P[b]) + W;
      const int64_t nsplit = std::min<int64_t>(p.splits, std::max<int64_t>(1, (n_all + p.kv_chunk - 1) / p.kv_chunk));
      const bool work = W > 0 && static_cast<int64_t>(qtile) * kRowsPerTile < static_cast<int64_t>(p.group) * W &&
                        split < nsplit;
      if (work) REQUIRE(seen[u] == 1);
    }
  }
  return hipSuccess;
}

hipError_t launch_edit_select(const EsParams &, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_threshold_update(const EsParams &, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_tail_entropy_scores(const float *, int64_t, int32_t, int32_t, float *, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_select_start_block(const float *, int32_t, int32_t, const int32_t *, int32_t, int32_t *,
                                     hipStream_t) {
  return hipSuccess;
}
hipError_t launch_refresh_blocks(const uint8_t *, int32_t, int32_t, int32_t, uint8_t *, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_kv_write(const KvWriteParams &, hipStream_t) { return hipSuccess; }

}  // namespace mbe
