// Ids partition without allocation: the same passes as ids_partition, with
// their workspace in a fixed device array of this library instead of a
// caller's buffer, for callers that cannot allocate device memory (code under
// HIP graph capture, serving loops, harnesses that forbid hipMalloc).
//
// The array is a file-scope __device__ variable: every GPU the library runs
// on holds its own copy, at its own address, until the process ends.  Host
// code never passes the variable's name to a kernel (on the host it is a
// stand-in, not a device address): the address is taken once per device
// with hipGetSymbolAddress, with that device current, and kept.
#include <hip/hip_runtime.h>

#include <mutex>

#include "recis_mi355x.h"
#include "rs_internal.h"

namespace {

// Workspace of ids_partition for at most RS_IDS_STATIC_MAX_IDS ids into at
// most 1024 shards (the largest case needs 53.5 MiB).
constexpr size_t kStaticBytes = size_t(54) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) uint8_t scratch[kStaticBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (null on failure).
void* scratch_ptr(int dev) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" rs_status ids_partition_static(const int64_t* values, int64_t n, int32_t nshards, uint64_t owner_seed,
                                          int64_t* keys_out, int64_t* shard_offsets, int32_t* inverse, int64_t* info,
                                          rs_stream stream) {
  if (n < 0 || n > RS_IDS_STATIC_MAX_IDS)
    return rs::set_last_error(RS_EINVAL, "n must be in [0, RS_IDS_STATIC_MAX_IDS] (2^20) for the no-allocation call");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return rs::set_last_error(RS_EHIP, "no current HIP device (or its ordinal is 64 or above)");
  }
  void* ws = scratch_ptr(dev);
  if (!ws) return rs::set_last_error(RS_EHIP, "hipGetSymbolAddress of the static workspace failed");
  // the workspace check inside ids_partition rejects a layout larger than
  // the array (it cannot happen for n <= RS_IDS_STATIC_MAX_IDS)
  return ids_partition(values, n, nshards, owner_seed, keys_out, shard_offsets, inverse, info, ws, kStaticBytes,
                       stream);
}
