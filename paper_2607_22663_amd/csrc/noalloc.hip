// mbe_threshold_update_noalloc: the threshold update for callers that cannot
// allocate device memory and hold no workspace of their own (code under HIP
// graph capture, tight serving loops, harnesses that forbid allocation).
//
// The update's kernels need scratch memory: each row's prediction between
// the row pass and the per-block step, plus per-chunk partial results when a
// row is reduced by several workgroups.  Here that scratch is a file-scope
// device array, one copy per GPU, alive until the process ends.  Its device
// address is looked up once per device (with that device current) on the
// first call there and kept; kernels always receive that address, never the
// host-side name of the array.  Every call on a GPU shares its array, so
// calls that overlap in time on one GPU (different streams, or host threads)
// race; calls on one stream run in order.  Nothing in the array has to start
// at zero: each call writes every prediction and partial before reading it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"
#include "mbe.h"

namespace {

constexpr size_t kScratchBytes = size_t(1) << 20;   // 1 MiB per GPU
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (looked up once per device).
mbe_status scratch_address(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return mbe::report(MBE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return mbe::report(MBE_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return mbe::report(MBE_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return MBE_OK;
}

}  // namespace

extern "C" {

mbe_status mbe_threshold_update_noalloc(const void *logits, int64_t rows, int64_t vocab, int64_t row_stride,
                                        const int32_t *cur_tokens, int32_t mask_id, int32_t block_size,
                                        float omega_mask, float omega_edit, int32_t *new_tokens, float *conf,
                                        uint8_t *action, uint8_t *block_changed, int32_t *changed_count,
                                        float *entropy, const int32_t *run_if_nonzero, void *stream) {
  size_t need = 0;
  mbe_status st = mbe::threshold_update_check(logits, rows, vocab, row_stride, cur_tokens, block_size, omega_mask,
                                              omega_edit, new_tokens, conf, action, block_changed, changed_count,
                                              run_if_nonzero, &need);
  if (st != MBE_OK || rows == 0) return st;
  if (need > kScratchBytes)
    return mbe::report(MBE_ERR_WORKSPACE,
                       "%lld rows x %lld vocab need %zu bytes of scratch, more than the static %zu "
                       "(use mbe_threshold_update with a workspace)",
                       static_cast<long long>(rows), static_cast<long long>(vocab), need, kScratchBytes);
  void *ws = nullptr;
  st = scratch_address(&ws);
  if (st != MBE_OK) return st;
  return mbe::threshold_update_launch(logits, rows, vocab, row_stride, cur_tokens, mask_id, block_size, omega_mask,
                                      omega_edit, new_tokens, conf, action, block_changed, changed_count, entropy,
                                      run_if_nonzero, ws, stream);
}

}  // extern "C"
