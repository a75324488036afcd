// Randomised host-side check of libmbe's C ABI, built with a host compiler
// under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU needed): the
// attention split planner, dispatch tables and workspace sizes over random
// ragged batches, and the edit-selection / threshold-update workspace sizes.
// For every case the size query and the call must agree: the call succeeds
// with exactly the queried workspace (and its plan passes the checks of the
// launcher stand-in) and fails with MBE_ERR_WORKSPACE with one byte less.
//
//   plan_fuzz <seed> <cases>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "mbe.h"

namespace fuzz {
extern const int32_t *host_P;
extern const int32_t *host_W;
extern size_t ws_bytes;
extern long launches;
extern long unit_tables;
}  // namespace fuzz

#define CHECK(c, ...)                                   \
  do {                                                  \
    if (!(c)) {                                         \
      std::fprintf(stderr, "case %ld: ", case_id);      \
      std::fprintf(stderr, __VA_ARGS__);                \
      std::fprintf(stderr, " [%s]\n", mbe_last_error()); \
      std::abort();                                     \
    }                                                   \
  } while (0)

static long case_id = 0;
static void *fake(uintptr_t a) { return reinterpret_cast<void *>(a); }

int main(int argc, char **argv) {
  const unsigned seed = argc > 1 ? static_cast<unsigned>(std::atoi(argv[1])) : 1u;
  const long cases = argc > 2 ? std::atol(argv[2]) : 2000;
  std::mt19937_64 rng(seed);
  auto U = [&](long lo, long hi) { return std::uniform_int_distribution<long>(lo, hi)(rng); };
  long splits_seen = 0, tables_seen = 0;
  for (case_id = 0; case_id < cases; ++case_id) {
    const int hkv = 1 << U(0, 3);
    const int G = 1 << U(0, 3);
    const int D = U(0, 1) ? 128 : 64;
    const int B = std::vector<int>{1, 8, 16, 32, 32, 32}[U(0, 5)];
    const int kmax = static_cast<int>(U(1, 8));
    const int shape = static_cast<int>(U(0, 3));
    const int batch = shape == 0 ? static_cast<int>(U(0, 3)) : shape == 1 ? static_cast<int>(U(1, 64))
                                                     : shape == 2 ? static_cast<int>(U(1, 300))
                                                                  : static_cast<int>(U(900, 1100));
    const long pmax = std::vector<long>{0, 64, 3000, 40000}[U(0, 3)];
    std::vector<int32_t> P(batch), W(batch);
    int32_t maxP = 0, maxW = 0;
    long total = 0;
    for (int b = 0; b < batch; ++b) {
      P[b] = static_cast<int32_t>(U(0, pmax));
      W[b] = static_cast<int32_t>(B * (U(0, 5) == 0 ? U(0, kmax) : kmax));
      maxP = std::max(maxP, P[b]);
      maxW = std::max(maxW, W[b]);
      total += W[b];
    }
    const bool bd = U(0, 4) == 0;                 // block_diffusion_attention: W_b = B
    if (bd) {
      for (int b = 0; b < batch; ++b) W[b] = B;
      maxW = B;
      total = static_cast<long>(batch) * B;
    }
    const int32_t bound_P = maxP + static_cast<int32_t>(U(0, 1) ? 0 : U(0, 100));
    const int32_t bound_W = bd ? B : maxW + B * static_cast<int32_t>(U(0, 1));
    mbe_paged_kv kv = {fake(0x10000), fake(0x20000), 1000, 16, hkv, D};
    mbe_attn_opts o = {};
    o.batch = batch;
    o.num_q_heads = hkv * G;
    o.max_pages_per_seq = (bound_P + bound_W + 15) / 16 + 1;
    o.total_q = static_cast<int32_t>(total);
    o.max_prefix_len = bound_P;
    o.max_window_len = bound_W;
    o.mask_mode = static_cast<int32_t>(U(0, 1));
    o.kv_split_tokens = U(0, 5) == 0 ? static_cast<int32_t>(64 * U(1, 40)) : 0;
    const bool host = U(0, 3) != 0;
    o.host_prefix_lens = host ? P.data() : nullptr;
    o.host_window_lens = host ? W.data() : nullptr;
    const size_t need = bd ? mbe_block_diffusion_workspace_size(&kv, &o, B)
                           : mbe_window_attention_workspace_size(&kv, &o);
    CHECK(need != static_cast<size_t>(-1), "size query rejected a valid shape");
    fuzz::host_P = host ? P.data() : nullptr;
    fuzz::host_W = host ? W.data() : nullptr;
    fuzz::ws_bytes = need;
    o.workspace = need ? fake(0x4000000) : nullptr;
    o.workspace_bytes = need;
    const long before = fuzz::launches;
    const mbe_status st = bd ? block_diffusion_attention(fake(0x30000), &kv, static_cast<const int32_t *>(fake(0x40000)),
                                                         static_cast<const int32_t *>(fake(0x50000)), B, fake(0x60000), &o)
                             : mbe_window_attention(fake(0x30000), &kv, static_cast<const int32_t *>(fake(0x40000)),
                                                    static_cast<const int32_t *>(fake(0x50000)),
                                                    static_cast<const int32_t *>(fake(0x70000)), B, fake(0x60000), &o);
    CHECK(st == MBE_OK, "call with the queried workspace failed: %d", static_cast<int>(st));
    CHECK(fuzz::launches == before + ((batch > 0 && total > 0) ? 1 : 0), "launch count");
    splits_seen += need > 0;
    if (need > 0) {
      o.workspace_bytes = need - 1;
      const mbe_status st2 = bd ? block_diffusion_attention(fake(0x30000), &kv, static_cast<const int32_t *>(fake(0x40000)),
                                                            static_cast<const int32_t *>(fake(0x50000)), B, fake(0x60000), &o)
                                : mbe_window_attention(fake(0x30000), &kv, static_cast<const int32_t *>(fake(0x40000)),
                                                       static_cast<const int32_t *>(fake(0x50000)),
                                                       static_cast<const int32_t *>(fake(0x70000)), B, fake(0x60000), &o);
      CHECK(st2 == MBE_ERR_WORKSPACE, "one byte short was accepted: %d", static_cast<int>(st2));
      CHECK(fuzz::launches == before + 1, "a rejected call launched");
    }
    tables_seen += host && batch > 1 && need > 0;

    // edit selection and threshold update sizes
    const int64_t rows = B * U(0, 700);
    const int64_t vocab = U(1, 200000);
    const size_t es = mbe_edit_select_workspace_size(rows, vocab);
    const size_t tu = mbe_threshold_update_workspace_size(rows, vocab);
    CHECK(es != static_cast<size_t>(-1) && tu != static_cast<size_t>(-1), "edit sizes");
    CHECK(rows == 0 || tu >= es + static_cast<size_t>(rows) * 4, "update workspace holds predictions and partials");
    if (rows > 0) {
      mbe_status s1 = mbe_edit_select(fake(0x80000), rows, vocab, vocab, static_cast<const int32_t *>(fake(0x90000)),
                                      0.9f, static_cast<int32_t *>(fake(0xa0000)), static_cast<float *>(fake(0xb0000)),
                                      static_cast<uint8_t *>(fake(0xc0000)), es ? fake(0x4000000) : nullptr, es, nullptr);
      CHECK(s1 == MBE_OK, "edit select with its workspace: %d", static_cast<int>(s1));
      if (es > 0) {
        s1 = mbe_edit_select(fake(0x80000), rows, vocab, vocab, static_cast<const int32_t *>(fake(0x90000)), 0.9f,
                             static_cast<int32_t *>(fake(0xa0000)), static_cast<float *>(fake(0xb0000)),
                             static_cast<uint8_t *>(fake(0xc0000)), fake(0x4000000), es - 1, nullptr);
        CHECK(s1 == MBE_ERR_WORKSPACE, "edit select one byte short");
      }
      mbe_status s2 = mbe_threshold_update(fake(0x80000), rows, vocab, vocab, static_cast<const int32_t *>(fake(0x90000)),
                                           3, B, 0.5f, 0.0f, static_cast<int32_t *>(fake(0xa0000)),
                                           static_cast<float *>(fake(0xb0000)), static_cast<uint8_t *>(fake(0xc0000)),
                                           static_cast<uint8_t *>(fake(0xd0000)), nullptr, nullptr, nullptr,
                                           fake(0x4000000), tu, nullptr);
      CHECK(s2 == MBE_OK, "threshold update with its workspace: %d", static_cast<int>(s2));
      s2 = mbe_threshold_update(fake(0x80000), rows, vocab, vocab, static_cast<const int32_t *>(fake(0x90000)), 3, B,
                                0.5f, 0.0f, static_cast<int32_t *>(fake(0xa0000)), static_cast<float *>(fake(0xb0000)),
                                static_cast<uint8_t *>(fake(0xc0000)), static_cast<uint8_t *>(fake(0xd0000)), nullptr,
                                nullptr, nullptr, fake(0x4000000), tu - 1, nullptr);
      CHECK(s2 == MBE_ERR_WORKSPACE, "threshold update one byte short");
    }
  }
  std::printf("plan_fuzz ok: %ld cases, %ld with split-KV workspaces, %ld ragged with host lengths, "
              "%ld host-placed dispatch tables\n", cases, splits_seen, tables_seen, fuzz::unit_tables);
  return 0;
}
