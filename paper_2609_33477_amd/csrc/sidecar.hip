// Anchor sidecar: the write path (destination table, prefill compaction,
// indexed copy; Section 5.1) and the read path (gather of the last k anchors
// into the packed replay batch; Section 5.2).  All of it is byte copying, so
// the roofline is HBM: the copies move 16-byte vectors, a wave per one or
// two rows, with every load of two rows in flight before their stores.
//
// Pool layout [n_blocks][n_layers][per_page][d]: one block per KV page, each
// anchored layer's per_page rows contiguous (d * elem_bytes bytes each).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "sr_internal.hpp"
#include "sr_sidecar.h"

namespace {

constexpr int kMaxLayers = 64;
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
constexpr int kWaves = 4;            // waves per workgroup of the copy kernels
constexpr int kScanThreads = 1024;   // the single-workgroup scans
constexpr int kScanPer = 64;         // entries per thread per pass of the compaction

// Copy two rows of `bytes` bytes (a multiple of 16) with the 64 lanes of a
// wave, 16 bytes per lane and step: all U steps of both rows are loaded
// before any is stored, so a wave keeps up to 2 U KB in flight; rows longer
// than U KB go in pieces.  Steps past the row's end load the row's first
// bytes again (cheap, and it keeps the loads unpredicated) and store
// nothing.  src1 = null copies one row.
template <int U>
__device__ __forceinline__ void wave_copy2(char* __restrict__ dst0, const char* __restrict__ src0,
                                           char* __restrict__ dst1, const char* __restrict__ src1, int bytes,
                                           int lane) {
  const char* s1 = src1 ? src1 : src0;
  for (int p = 0; p < bytes; p += U * 1024) {
    u32x4 v0[U], v1[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int o = p + u * 1024 + lane * 16;
      const int oc = o < bytes ? o : 0;
      v0[u] = *reinterpret_cast<const u32x4*>(src0 + oc);
      v1[u] = *reinterpret_cast<const u32x4*>(s1 + oc);
    }
    // every loaded value is live here, so no load sinks to its store
#pragma unroll
    for (int u = 0; u < U; ++u) asm volatile("" : "+v"(v0[u]), "+v"(v1[u]));
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int o = p + u * 1024 + lane * 16;
      if (o < bytes) {
        *reinterpret_cast<u32x4*>(dst0 + o) = v0[u];
        if (src1) *reinterpret_cast<u32x4*>(dst1 + o) = v1[u];
      }
    }
  }
}

// The number of 1 KB wave steps per piece: a whole row up to 8 KB.
inline int copy_steps(int row_bytes) {
  const int u = (row_bytes + 1023) / 1024;
  return u < 1 ? 1 : (u > 8 ? 8 : u);
}

// Inclusive sum of x over the 64 lanes of a wave.
__device__ __forceinline__ int wave_inclusive_sum(int x, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  return x;
}

// Exclusive offset of each wave's total inside the workgroup, and the
// workgroup's total, from the per-wave totals in `wsum`.
__device__ __forceinline__ void wave_offsets(const int* wsum, int w, int& before, int& total) {
  before = 0;
  total = 0;
  for (int j = 0; j < kScanThreads / 64; ++j) {
    if (j < w) before += wsum[j];
    total += wsum[j];
  }
}

// --------------------------------------------------------- compaction (5.1)
// One workgroup: thread t of a pass looks at entries c0 + 64 t .. + 63
// (16-byte loads where the table is aligned, so a 64K-token step is one
// pass) and writes the indices of those with a destination at its exclusive
// offset.
__global__ __launch_bounds__(kScanThreads) void compact_kernel(const int32_t* __restrict__ dest, int32_t n,
                                                              int32_t* __restrict__ sel,
                                                              int32_t* __restrict__ n_sel, bool vec) {
  __shared__ int wsum[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int base = 0;
  for (int64_t c0 = 0; c0 < n; c0 += (int64_t)kScanThreads * kScanPer) {
    const int64_t i0 = c0 + (int64_t)tid * kScanPer;
    uint64_t flags = 0;
    if (vec && i0 + kScanPer <= n) {
#pragma unroll
      for (int k = 0; k < kScanPer; k += 4) {
        const int4 v = *reinterpret_cast<const int4*>(dest + i0 + k);
        flags |= (uint64_t)(v.x >= 0) << k | (uint64_t)(v.y >= 0) << (k + 1) | (uint64_t)(v.z >= 0) << (k + 2) |
                 (uint64_t)(v.w >= 0) << (k + 3);
      }
    } else {
      for (int k = 0; k < kScanPer; ++k)
        if (i0 + k < n && dest[i0 + k] >= 0) flags |= (uint64_t)1 << k;
    }
    const int cnt = __builtin_popcountll(flags);
    const int incl = wave_inclusive_sum(cnt, lane);
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int before, total;
    wave_offsets(wsum, w, before, total);
    int pos = base + before + incl - cnt;
    while (flags) {
      const int k = __builtin_ctzll(flags);
      flags &= flags - 1;
      sel[pos++] = (int32_t)(i0 + k);
    }
    base += total;
    __syncthreads();   // wsum is rewritten by the next pass
  }
  if (tid == 0) *n_sel = base;
}

// ------------------------------------------------------- indexed copy (5.1)
struct WriteArgs {
  char* pool;
  int32_t n_layers, per_page, row_bytes, n_tokens;
  const int32_t* dest;
  const int32_t* sel;     // work list, or null: every token
  const int32_t* n_sel;
  const char* hidden[kMaxLayers];
};

template <int U>
__global__ __launch_bounds__(64 * kWaves) void write_kernel(WriteArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * kWaves;
  const int n = a.sel ? *a.n_sel : a.n_tokens;
  for (int k = wave; k < n; k += n_waves) {
    const int i = __builtin_amdgcn_readfirstlane(a.sel ? a.sel[k] : k);
    const int row = __builtin_amdgcn_readfirstlane(a.dest[i]);
    if (row < 0) continue;
    const int64_t blk = row / a.per_page, slot = row % a.per_page;
    for (int l = 0; l < a.n_layers; l += 2) {
      const bool two = l + 1 < a.n_layers;
      char* dst = a.pool + ((blk * a.n_layers + l) * a.per_page + slot) * a.row_bytes;
      const char* src = a.hidden[l] + (int64_t)i * a.row_bytes;
      wave_copy2<U>(dst, src, two ? dst + (int64_t)a.per_page * a.row_bytes : nullptr,
                 two ? a.hidden[l + 1] + (int64_t)i * a.row_bytes : nullptr, a.row_bytes, lane);
    }
  }
}

// ------------------------------------------------------------ gather (5.2)
// cu_seqlens = prefix sums of n_anchors, one workgroup.
__global__ __launch_bounds__(kScanThreads) void seqlens_kernel(const int32_t* __restrict__ n_anchors, int32_t n,
                                                              int32_t* __restrict__ cu) {
  __shared__ int wsum[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) cu[0] = 0;
  int base = 0;
  for (int c0 = 0; c0 < n; c0 += kScanThreads) {
    const int i = c0 + tid;
    const int x = i < n ? n_anchors[i] : 0;
    const int incl = wave_inclusive_sum(x, lane);
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int before, total;
    wave_offsets(wsum, w, before, total);
    if (i < n) cu[i + 1] = base + before + incl;
    base += total;
    __syncthreads();
  }
}

struct GatherArgs {
  const char* pool;
  int32_t n_layers, per_page, row_bytes, n_req, n_out;
  int64_t t_cap;
  const int32_t* block_table;
  const int32_t* block_cu;
  const int32_t* anchor_first;
  const int32_t* cu;
  char* out[kMaxLayers];
  int32_t layer[kMaxLayers];
};

constexpr int kRowsPerWave = 1;

// A wave copies kRowsPerWave consecutive output rows: it finds the first
// row's request by binary search over cu_seqlens, then steps forward.
template <int U>
__global__ __launch_bounds__(64 * kWaves) void gather_kernel(GatherArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int64_t total = a.cu[a.n_req] < a.t_cap ? a.cu[a.n_req] : a.t_cap;
  const int64_t row0 = wave * kRowsPerWave;
  if (row0 >= total) return;
  // request r with cu[r] <= row0 < cu[r + 1] (empty requests are skipped)
  int lo = 0, hi = a.n_req - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.cu[mid] <= row0) lo = mid;
    else hi = mid - 1;
  }
  int r = __builtin_amdgcn_readfirstlane(lo);
  int r_end = a.cu[r + 1];
  for (int64_t row = row0; row < row0 + kRowsPerWave && row < total; ++row) {
    while (row >= r_end) {
      ++r;
      r_end = a.cu[r + 1];
    }
    const int j = __builtin_amdgcn_readfirstlane(a.anchor_first[r] + (int)(row - a.cu[r]));
    const int64_t blk = __builtin_amdgcn_readfirstlane(a.block_table[a.block_cu[r] + j / a.per_page]);
    const int slot = j % a.per_page;
    const char* base = a.pool + (blk * a.n_layers * a.per_page + slot) * a.row_bytes;
    const int64_t lstride = (int64_t)a.per_page * a.row_bytes;   // one layer's rows in a block
    for (int o = 0; o < a.n_out; o += 2) {
      const bool two = o + 1 < a.n_out;
      wave_copy2<U>(a.out[o] + row * a.row_bytes, base + a.layer[o] * lstride,
                 two ? a.out[o + 1] + row * a.row_bytes : nullptr, two ? base + a.layer[o + 1] * lstride : nullptr,
                 a.row_bytes, lane);
    }
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sr_status check_sidecar(const sr_sidecar* sc) {
  if (!sc || !sc->pool) return SR_ERR_NULL_ARG;
  if (sc->n_blocks < 1 || sc->n_layers < 1 || sc->n_layers > kMaxLayers || sc->per_page < 1 ||
      sc->per_page > 64 || sc->d < 1)
    return SR_ERR_BAD_SHAPE;
  if (sc->elem_bytes != 2 && sc->elem_bytes != 4) return SR_ERR_UNSUPPORTED_DTYPE;
  if (((int64_t)sc->d * sc->elem_bytes) % 16 != 0 || (int64_t)sc->d * sc->elem_bytes > (1 << 24))
    return SR_ERR_BAD_SHAPE;
  if (!aligned16(sc->pool)) return SR_ERR_MISALIGNED;
  return SR_OK;
}

// Launch through the library's timing and failed-launch bookkeeping.
template <typename F>
sr_status launch(int kind, hipStream_t s, F&& f) {
  return sr::timed_call(kind, s, [&] {
    f();
    return hipGetLastError();
  }) == hipSuccess ? SR_OK : SR_ERR_HIP;
}

}  // namespace

extern "C" {

sr_status sr_anchor_dest_table(const int32_t* positions, const int32_t* token_req, int32_t n_tokens,
                               const int32_t* page_table, const int32_t* page_cu, int32_t n_req,
                               int32_t page_size, int32_t per_page, int32_t* dest) {
  if (n_tokens < 0 || n_req < 0 || page_size < 1 || per_page < 1 || per_page > page_size) return SR_ERR_BAD_SHAPE;
  if (n_tokens == 0) return SR_OK;
  if (!positions || !token_req || !page_cu || !dest || n_req == 0) return SR_ERR_NULL_ARG;
  if (page_cu[0] != 0) return SR_ERR_BAD_SHAPE;
  for (int32_t r = 0; r < n_req; ++r)
    if (page_cu[r + 1] < page_cu[r]) return SR_ERR_BAD_SHAPE;
  if (page_cu[n_req] > 0 && !page_table) return SR_ERR_NULL_ARG;
  for (int32_t i = 0; i < n_tokens; ++i)
    if (token_req[i] < 0 || token_req[i] >= n_req || positions[i] < 0) return SR_ERR_BAD_SHAPE;
  const int32_t first = page_size - per_page;   // first anchor row of a page
  for (int32_t i = 0; i < n_tokens; ++i) {
    const int32_t t = positions[i], r = token_req[i];
    const int32_t in_page = t % page_size, q = t / page_size;
    int32_t row = -1;
    if (in_page >= first && q < page_cu[r + 1] - page_cu[r]) {
      const int32_t blk = page_table[page_cu[r] + q];
      if (blk >= 0) row = blk * per_page + (in_page - first);
    }
    dest[i] = row;
  }
  return SR_OK;
}

sr_status sr_anchor_compact(const int32_t* dest, int32_t n_tokens, int32_t* sel, int32_t* n_sel, void* stream) {
  if (n_tokens < 0 || n_tokens > (1 << 30)) return SR_ERR_BAD_SHAPE;
  if (!n_sel || (n_tokens > 0 && (!dest || !sel))) return SR_ERR_NULL_ARG;
  hipStream_t s = (hipStream_t)stream;
  return launch(SR_KERNEL_ANCHOR_COMPACT, s, [&] {
    hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(kScanThreads), 0, s, dest, n_tokens, sel, n_sel,
                       aligned16(dest));
  });
}

sr_status sr_anchor_write(const sr_sidecar* sc, const void* const* hidden, int32_t n_tokens, const int32_t* dest,
                          const int32_t* sel, const int32_t* n_sel, void* stream) {
  const sr_status st = check_sidecar(sc);
  if (st != SR_OK) return st;
  if (n_tokens < 0) return SR_ERR_BAD_SHAPE;
  if (n_tokens == 0) return SR_OK;
  if (!hidden || !dest || (sel && !n_sel)) return SR_ERR_NULL_ARG;
  WriteArgs a{};
  a.pool = static_cast<char*>(sc->pool);
  a.n_layers = sc->n_layers;
  a.per_page = sc->per_page;
  a.row_bytes = sc->d * sc->elem_bytes;
  a.n_tokens = n_tokens;
  a.dest = dest;
  a.sel = sel;
  a.n_sel = n_sel;
  for (int l = 0; l < sc->n_layers; ++l) {
    if (!hidden[l]) return SR_ERR_NULL_ARG;
    if (!aligned16(hidden[l])) return SR_ERR_MISALIGNED;
    a.hidden[l] = static_cast<const char*>(hidden[l]);
  }
  const int waves = n_tokens < 8192 ? n_tokens : 8192;
  hipStream_t s = (hipStream_t)stream;
  const dim3 grid((waves + kWaves - 1) / kWaves), block(64 * kWaves);
  return launch(SR_KERNEL_ANCHOR_WRITE, s, [&] {
    switch (copy_steps(a.row_bytes)) {
      case 1: hipLaunchKernelGGL(write_kernel<1>, grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL(write_kernel<2>, grid, block, 0, s, a); break;
      case 3: hipLaunchKernelGGL(write_kernel<3>, grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL(write_kernel<4>, grid, block, 0, s, a); break;
      case 5: hipLaunchKernelGGL(write_kernel<5>, grid, block, 0, s, a); break;
      case 6: hipLaunchKernelGGL(write_kernel<6>, grid, block, 0, s, a); break;
      case 7: hipLaunchKernelGGL(write_kernel<7>, grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL(write_kernel<8>, grid, block, 0, s, a); break;
    }
  });
}

sr_status sr_anchor_gather(const sr_sidecar* sc, int32_t n_req, const int32_t* block_table,
                           const int32_t* block_cu, const int32_t* anchor_first, const int32_t* n_anchors,
                           const int32_t* layers, int32_t n_out, void* const* out, int64_t t_cap,
                           int32_t* cu_seqlens, void* stream) {
  const sr_status st = check_sidecar(sc);
  if (st != SR_OK) return st;
  if (n_req < 0 || n_req > 65536 || n_out < 1 || n_out > kMaxLayers || t_cap < 0) return SR_ERR_BAD_SHAPE;
  if (!cu_seqlens || !layers || !out) return SR_ERR_NULL_ARG;
  if (n_req > 0 && (!block_table || !block_cu || !anchor_first || !n_anchors)) return SR_ERR_NULL_ARG;
  GatherArgs a{};
  a.pool = static_cast<const char*>(sc->pool);
  a.n_layers = sc->n_layers;
  a.per_page = sc->per_page;
  a.row_bytes = sc->d * sc->elem_bytes;
  a.n_req = n_req;
  a.n_out = n_out;
  a.t_cap = t_cap;
  a.block_table = block_table;
  a.block_cu = block_cu;
  a.anchor_first = anchor_first;
  a.cu = cu_seqlens;
  for (int o = 0; o < n_out; ++o) {
    if (layers[o] < 0 || layers[o] >= sc->n_layers) return SR_ERR_BAD_SHAPE;
    if (!out[o] && t_cap > 0) return SR_ERR_NULL_ARG;
    if (!aligned16(out[o])) return SR_ERR_MISALIGNED;
    a.out[o] = static_cast<char*>(out[o]);
    a.layer[o] = layers[o];
  }
  hipStream_t s = (hipStream_t)stream;
  if (launch(SR_KERNEL_ANCHOR_SEQLENS, s, [&] {
        hipLaunchKernelGGL(seqlens_kernel, dim3(1), dim3(kScanThreads), 0, s, n_anchors, n_req, cu_seqlens);
      }) != SR_OK)
    return SR_ERR_HIP;
  if (n_req == 0 || t_cap == 0) return SR_OK;
  const int64_t waves = (t_cap + kRowsPerWave - 1) / kRowsPerWave;
  const dim3 grid((unsigned)((waves + kWaves - 1) / kWaves)), block(64 * kWaves);
  return launch(SR_KERNEL_ANCHOR_GATHER, s, [&] {
    switch (copy_steps(a.row_bytes)) {
      case 1: hipLaunchKernelGGL(gather_kernel<1>, grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL(gather_kernel<2>, grid, block, 0, s, a); break;
      case 3: hipLaunchKernelGGL(gather_kernel<3>, grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL(gather_kernel<4>, grid, block, 0, s, a); break;
      case 5: hipLaunchKernelGGL(gather_kernel<5>, grid, block, 0, s, a); break;
      case 6: hipLaunchKernelGGL(gather_kernel<6>, grid, block, 0, s, a); break;
      case 7: hipLaunchKernelGGL(gather_kernel<7>, grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL(gather_kernel<8>, grid, block, 0, s, a); break;
    }
  });
}

}  // extern "C"
