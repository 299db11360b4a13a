// Allocation-free paged prefill attention: ilpc_paged_prefill_attn with a
// workspace that is a static device array of this library instead of a
// buffer the caller allocates.  For callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).
//
// The array holds the attention kernel's work-queue counters in its first 64
// bytes (zero when the code object is loaded; every call's last workgroup
// leaves them zero again) and, after them, room for the split decode kernel's
// partial results.  Each GPU holds its own copy until the process ends, and
// every call on a GPU shares it, so calls that may overlap on one GPU race.
// In host code `scratch` names only the host-side stand-in of the device
// symbol, never device memory: kernels get the address hipGetSymbolAddress
// returns for the current device, looked up once per device.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <mutex>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace {

constexpr size_t kScratchBytes = 256 + (size_t(8) << 20);
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

// Device address of `scratch` on the current device, looked up with that
// device current the first time a call runs on it; nullptr (message set) on
// failure.
void* scratch_address(const char* fn) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    ilpc::set_error(ILPC_EHIP, "%s: no usable current device (%s)", fn, hipGetErrorString(e));
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      ilpc::set_error(ILPC_EHIP, "%s: hipGetSymbolAddress(scratch) on device %d failed: %s", fn, dev,
                      hipGetErrorString(e));
      return nullptr;
    }
    addr[dev] = p;
  }
  return addr[dev];
}

}  // namespace

extern "C" int ilpc_paged_prefill_attn_noalloc(const uint16_t* q, const uint16_t* k_pool,
                                               const uint16_t* v_pool, int32_t num_blocks,
                                               const int32_t* block_tables, int32_t max_blocks,
                                               const int32_t* cu_q, const int32_t* seq_lens, int32_t B,
                                               int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                               int32_t block_size, float softmax_scale, uint16_t* out,
                                               void* stream) {
  // Argument errors are reported by ilpc_paged_prefill_attn before anything
  // runs; an empty batch needs no scratch.
  if (B == 0 || max_q_len == 0)
    return ilpc_paged_prefill_attn(q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                                   max_q_len, Hq, Hkv, D, block_size, softmax_scale, out, nullptr, 0, stream);
  void* ws = scratch_address("ilpc_paged_prefill_attn_noalloc");
  if (!ws) return ILPC_EHIP;
  return ilpc_paged_prefill_attn(q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                                 max_q_len, Hq, Hkv, D, block_size, softmax_scale, out, ws, kScratchBytes, stream);
}
