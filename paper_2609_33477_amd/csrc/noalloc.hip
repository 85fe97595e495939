// sr_replay_state_noalloc: the replay of sr_replay_state() for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc).  Its workspace is a file-scope
// device array of SR_NOALLOC_SCRATCH_BYTES, one copy per GPU, held until the
// process ends.
//
// Host code never passes the array's name to a kernel: in host code that name
// is a host-side stand-in, not a device address.  The first call on a device
// resolves the array's address on that device with hipGetSymbolAddress (with
// the device current) and keeps it per device; every later use goes through
// that pointer.  The replay's kernels write every workspace byte they read
// within a call (the table check's flag word, row info, k, v, log-decay and
// beta planes), so nothing needs clearing between calls.  Calls that overlap
// on one GPU share the array and race; calls on one GPU must be ordered (one
// stream, or explicit events).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "sr_replay.h"

namespace {

constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[SR_NOALLOC_SCRATCH_BYTES];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// The scratch array's device address on the current device, resolved once
// per device.  nullptr on a HIP error.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" sr_status sr_replay_state_noalloc(const sr_shape* shape, int32_t n_layers, const sr_layer* layers,
                                             int32_t n_segments, int64_t t_total, const int32_t* cu_seqlens,
                                             const int32_t* slot_ids, int32_t n_slots, int32_t* varlen_status,
                                             void* stream) {
  size_t need = 0;
  const sr_status st = sr_replay_workspace_size(shape, n_layers, t_total, &need);
  if (st != SR_OK) return st;
  if (need > (size_t)SR_NOALLOC_SCRATCH_BYTES) return SR_ERR_WORKSPACE_TOO_SMALL;
  if (!layers) return SR_ERR_NULL_ARG;
  void* ws = scratch_on_current_device();
  if (!ws) return SR_ERR_HIP;
  return sr_replay_state(shape, n_layers, layers, n_segments, t_total, cu_seqlens, slot_ids, n_slots, varlen_status,
                         ws, (size_t)SR_NOALLOC_SCRATCH_BYTES, stream);
}
