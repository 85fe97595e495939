// Device check of a replay call's varlen tables (Section 5.2: the pipeline is
// fail-closed; a bad input is treated as a cache miss, never written
// through).  One workgroup reads cu_seqlens [B + 1] and slot_ids [B] and
// writes 0 or a mask of sr_varlen_error bits to a flag word; every later
// kernel of the call reads that word first and exits if it is non-zero, so a
// table that would send rows or states out of their buffers makes the call
// write nothing.  Distinct live slots are checked with a bitmap of n_slots
// bits in LDS.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "sr_internal.hpp"
#include "sr_replay.h"

namespace sr {

constexpr int kThreads = 1024;
constexpr int kWords = SR_MAX_SLOTS / 32;   // 64 KiB of LDS

// The checks of segment b of B that need no other segment: everything but
// duplicate slots.  Shared by the device kernel and the host twin.
__host__ __device__ inline int32_t segment_mask(int32_t b, int32_t B, int32_t c0, int32_t c1, int64_t T, int32_t s,
                                                int32_t n_slots) {
  int32_t m = 0;
  if (b == 0 && c0 != 0) m |= SR_VARLEN_BAD_START;
  if (c1 < c0) m |= SR_VARLEN_NOT_MONOTONE;
  if (b == B - 1 && (int64_t)c1 != T) m |= SR_VARLEN_BAD_TOTAL;
  if (s >= n_slots) m |= SR_VARLEN_SLOT_RANGE;
  return m;
}

// The check itself, by one workgroup of kThreads.
__device__ __forceinline__ void check_tables(const int32_t* __restrict__ cu, const int32_t* __restrict__ slot_ids,
                                             int32_t B, int64_t T, int32_t n_slots, int32_t* flag, int32_t* status) {
  __shared__ uint32_t seen[kWords];
  __shared__ int32_t bad;
  const int words = (n_slots + 31) >> 5;
  for (int i = threadIdx.x; i < words; i += kThreads) seen[i] = 0u;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  int32_t mine = 0;
  for (int b = threadIdx.x; b < B; b += kThreads) {
    const int32_t s = slot_ids ? slot_ids[b] : b;
    mine |= segment_mask(b, B, cu[b], cu[b + 1], T, s, n_slots);
    if (s >= 0 && s < n_slots) {
      const uint32_t bit = 1u << (s & 31);
      if (atomicOr(&seen[s >> 5], bit) & bit) mine |= SR_VARLEN_SLOT_DUPLICATE;
    }
  }
  if (mine) atomicOr(&bad, mine);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (flag) *flag = bad;
    if (status) *status = bad;
  }
}

__global__ __launch_bounds__(kThreads) void validate_varlen_kernel(const int32_t* __restrict__ cu,
                                                                  const int32_t* __restrict__ slot_ids, int32_t B,
                                                                  int64_t T, int32_t n_slots, int32_t* flag,
                                                                  int32_t* status) {
  check_tables(cu, slot_ids, B, T, n_slots, flag, status);
}

// The check (block B) in one launch with the per-row segment info the fused
// projection reads (block b < B: segment b's rows).  The info is scratch in
// the call's workspace: it is written whatever the check finds, its rows
// clamped to [0, T), and nothing that reads it runs unless the check passed.
__global__ __launch_bounds__(kThreads) void validate_rows_kernel(const int32_t* __restrict__ cu,
                                                                 const int32_t* __restrict__ slot_ids, int32_t B,
                                                                 int64_t T, int32_t n_slots, int32_t* flag,
                                                                 int32_t* status, RowInfo* __restrict__ info) {
  if ((int)blockIdx.x == B) {
    check_tables(cu, slot_ids, B, T, n_slots, flag, status);
    return;
  }
  const int b = blockIdx.x;
  const int32_t s0 = cu[b], s1 = cu[b + 1];
  const int32_t slot = slot_ids ? slot_ids[b] : b;
  const int64_t lo = s0 < 0 ? 0 : s0, hi = (int64_t)s1 < T ? s1 : T;
  for (int64_t t = lo + threadIdx.x; t < hi; t += kThreads) {
    RowInfo v;
    v.pos = (int32_t)(t - s0);
    v.rem = (int32_t)(s1 - t);
    v.slot = slot;
    v.seg = b;
    info[t] = v;
  }
}

hipError_t launch_validate_rows(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, int64_t T,
                                int32_t n_slots, int32_t* flag, int32_t* status, RowInfo* info, hipStream_t s) {
  hipLaunchKernelGGL(validate_rows_kernel, dim3(n_seg + 1), dim3(kThreads), 0, s, cu, slot_ids, n_seg, T, n_slots,
                     flag, status, info);
  return hipGetLastError();
}

hipError_t launch_validate(const int32_t* cu, const int32_t* slot_ids, int32_t n_seg, int64_t T, int32_t n_slots,
                           int32_t* flag, int32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(validate_varlen_kernel, dim3(1), dim3(kThreads), 0, s, cu, slot_ids, n_seg, T, n_slots, flag,
                     status);
  return hipGetLastError();
}

}  // namespace sr

extern "C" sr_status sr_validate_varlen_host(const int32_t* cu_seqlens, const int32_t* slot_ids,
                                             int32_t n_segments, int64_t t_total, int32_t n_slots, int32_t* mask) {
  if (!cu_seqlens || !mask) return SR_ERR_NULL_ARG;
  if (n_segments < 1 || t_total < 0 || n_slots < 0 || n_slots > SR_MAX_SLOTS) return SR_ERR_BAD_SHAPE;
  std::vector<uint8_t> seen((size_t)n_slots, 0);
  int32_t m = 0;
  for (int32_t b = 0; b < n_segments; ++b) {
    const int32_t s = slot_ids ? slot_ids[b] : b;
    m |= sr::segment_mask(b, n_segments, cu_seqlens[b], cu_seqlens[b + 1], t_total, s, n_slots);
    if (s >= 0 && s < n_slots) {
      if (seen[s]) m |= SR_VARLEN_SLOT_DUPLICATE;
      seen[s] = 1;
    }
  }
  *mask = m;
  return SR_OK;
}

extern "C" sr_status sr_validate_varlen(const int32_t* cu_seqlens, const int32_t* slot_ids, int32_t n_segments,
                                        int64_t t_total, int32_t n_slots, int32_t* status, void* stream) {
  if (!cu_seqlens || !status) return SR_ERR_NULL_ARG;
  if (n_segments < 1 || t_total < 0 || n_slots < 0 || n_slots > SR_MAX_SLOTS) return SR_ERR_BAD_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = sr::timed_call(SR_KERNEL_VALIDATE, s, [&] {
    return sr::launch_validate(cu_seqlens, slot_ids, n_segments, t_total, n_slots, nullptr, status, s);
  });
  return e == hipSuccess ? SR_OK : SR_ERR_HIP;
}
