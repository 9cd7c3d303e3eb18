// The allocation-free variant of augtree_tree_bwd: its workspace (the tile
// schedules and D = rowsum(dO * O) of every row) is a fixed device array of
// this library instead of a caller buffer, so a call allocates nothing.
//
// Each GPU the library runs on holds its own copy of the array from the
// first call on it until the process ends. Host code never uses the array's
// name as an address: at the first call on a device (with that device
// current) the device address of that GPU's copy is looked up once with
// hipGetSymbolAddress and kept per device. Nothing in the array needs to
// start at zero (every call writes the schedule it reads and every D value
// before it is read). Calls that overlap on one GPU share the array and race.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "../../include/augtree.h"
#include "internal.h"

namespace augtree {
namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;  // 64 MiB

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// The current device's copy of the array (looked up once per device).
int scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail_status(AUGTREE_ERR_HIP, "allocation-free entry point: no usable current device");
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail_status(AUGTREE_ERR_HIP, "allocation-free entry point: hipGetSymbolAddress of the scratch array "
                                            "failed");
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return AUGTREE_OK;
}

}  // namespace
}  // namespace augtree

extern "C" {

size_t augtree_noalloc_scratch_bytes(void) { return augtree::kScratchBytes; }

int augtree_tree_bwd_noalloc(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p,
                             const uint16_t* v_p, const uint16_t* o_p, const float* lse_p, const uint16_t* do_p,
                             const uint16_t* q_r, const uint16_t* k_r, const uint16_t* v_r, const uint16_t* o_r,
                             const float* lse_r, const uint16_t* do_r, uint16_t* dq_p, uint16_t* dk_p,
                             uint16_t* dv_p, float* dkv_p_f32, uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r,
                             void* stream) {
  return augtree::tree_bwd_impl(grp, q_p, k_p, v_p, o_p, lse_p, do_p, q_r, k_r, v_r, o_r, lse_r, do_r, dq_p, dk_p,
                                dv_p, dkv_p_f32, dq_r, dk_r, dv_r, augtree::scratch_of_current_device, nullptr,
                                augtree::kScratchBytes, stream);
}

}  // extern "C"
