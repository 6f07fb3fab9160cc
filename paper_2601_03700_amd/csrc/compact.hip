// Active-index update of Appendix I: stable split of the active list by the
// exit flags into the rows that continue and the rows that exit.
//
// Small lists (the per-layer case: at most a few ten thousand rows) use one
// 1024-thread workgroup that walks the list in rounds of 4096 entries: each
// thread takes 4 consecutive entries (one 4-byte flag load, one 16-byte row
// load), counts its exits, and a wave scan (shuffles) plus a 16-entry LDS
// scan over the waves gives every thread its output offsets.  Larger lists
// use three passes over 16K-entry tiles (count, scan of tile counts, scatter)
// with the same in-tile scheme.  Both keep the input order.
#include "common.h"

namespace adept {
namespace {

constexpr int kThreads = 1024;
constexpr int kItems = 4;
constexpr int kRound = kThreads * kItems;      // entries per round
constexpr int kTileRounds = 4;                 // multi-pass tile = 16K entries
constexpr int kTile = kRound * kTileRounds;
constexpr int kSingleMax = 1 << 16;            // lists up to this use one workgroup

// Inclusive scan of v over the workgroup; returns the exclusive prefix and
// writes the workgroup total to *total.  `sh` holds >= 32 ints.
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      const int t = sh[w];
      sh[w] = run;
      run += t;
    }
    sh[kThreads / 64] = run;
  }
  __syncthreads();
  const int excl = sh[wave] + x - v;
  *total = sh[kThreads / 64];
  __syncthreads();
  return excl;
}

// Processes entries [start, end) of the list, writing kept rows at
// next[keep_base + ...] and exited rows at exited[exit_base + ...].
__device__ __forceinline__ void split_range(int start, int end, int layer,
                                            const uint8_t* __restrict__ flags,
                                            const int32_t* __restrict__ active,
                                            int32_t* __restrict__ next,
                                            int32_t* __restrict__ exited,
                                            int32_t* __restrict__ exit_layer, int* keep_base,
                                            int* exit_base, int* sh) {
  for (int r0 = start; r0 < end; r0 += kRound) {
    const int e0 = r0 + threadIdx.x * kItems;
    uint8_t f[kItems];
    int32_t rw[kItems];
    if (e0 + kItems <= end) {
      const uint32_t fw = *reinterpret_cast<const uint32_t*>(flags + e0);
      const int4 rv = *reinterpret_cast<const int4*>(active + e0);
      f[0] = fw & 0xff; f[1] = (fw >> 8) & 0xff; f[2] = (fw >> 16) & 0xff; f[3] = fw >> 24;
      rw[0] = rv.x; rw[1] = rv.y; rw[2] = rv.z; rw[3] = rv.w;
    } else {
#pragma unroll
      for (int q = 0; q < kItems; ++q) {
        const bool ok = e0 + q < end;
        f[q] = (ok && flags[e0 + q]) ? 1 : 0;
        rw[q] = ok ? active[e0 + q] : -1;
      }
    }
    int n_ex = 0, n_keep = 0;
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
      const bool valid = e0 + q < end;
      n_ex += (valid && f[q]) ? 1 : 0;
      n_keep += (valid && !f[q]) ? 1 : 0;
    }
    int tot_ex, tot_keep;
    int off_ex = block_exclusive_scan(n_ex, sh, &tot_ex);
    int off_keep = block_exclusive_scan(n_keep, sh, &tot_keep);
    off_ex += *exit_base;
    off_keep += *keep_base;
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
      if (e0 + q >= end) break;
      if (f[q]) {
        exited[off_ex++] = rw[q];
        exit_layer[rw[q]] = layer;
      } else {
        next[off_keep++] = rw[q];
      }
    }
    *exit_base += tot_ex;
    *keep_base += tot_keep;
  }
}

__global__ __launch_bounds__(kThreads) void compact_single(
    int layer, const uint8_t* __restrict__ flags, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active, int32_t* __restrict__ next, int32_t* __restrict__ n_next,
    int32_t* __restrict__ exited, int32_t* __restrict__ n_exited,
    int32_t* __restrict__ exit_layer, int max_n) {
  __shared__ int sh[kThreads / 64 + 1];
  const int n = min(*n_active, max_n);
  int keep = 0, ex = 0;
  split_range(0, n, layer, flags, active, next, exited, exit_layer, &keep, &ex, sh);
  if (threadIdx.x == 0) {
    *n_next = keep;
    *n_exited = ex;
  }
}

// pass 1: exits per tile
__global__ __launch_bounds__(kThreads) void compact_count(const uint8_t* __restrict__ flags,
                                                          const int32_t* __restrict__ n_active,
                                                          int32_t* __restrict__ tile_ex,
                                                          int max_n) {
  __shared__ int sh[kThreads / 64 + 1];
  const int n = min(*n_active, max_n);
  const int start = blockIdx.x * kTile;
  if (start >= n) return;
  const int end = min(n, start + kTile);
  int cnt = 0;
  for (int e = start + threadIdx.x; e < end; e += kThreads) cnt += flags[e] ? 1 : 0;
  int tot;
  block_exclusive_scan(cnt, sh, &tot);
  if (threadIdx.x == 0) tile_ex[blockIdx.x] = tot;
}

// pass 2: exclusive scan of the tile counts (one workgroup), totals
__global__ __launch_bounds__(kThreads) void compact_scan(const int32_t* __restrict__ n_active,
                                                         int32_t* __restrict__ tile_ex,
                                                         int32_t* __restrict__ n_next,
                                                         int32_t* __restrict__ n_exited,
                                                         int max_n) {
  __shared__ int sh[kThreads / 64 + 1];
  const int n = min(*n_active, max_n);
  const int tiles = (n + kTile - 1) / kTile;
  int carry = 0;
  for (int t0 = 0; t0 < tiles; t0 += kThreads) {
    const int t = t0 + threadIdx.x;
    const int v = t < tiles ? tile_ex[t] : 0;
    int tot;
    const int ex = block_exclusive_scan(v, sh, &tot);
    if (t < tiles) tile_ex[t] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    *n_exited = carry;
    *n_next = n - carry;
  }
}

// pass 3: scatter each tile from its offsets
__global__ __launch_bounds__(kThreads) void compact_scatter(
    int layer, const uint8_t* __restrict__ flags, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active, const int32_t* __restrict__ tile_ex,
    int32_t* __restrict__ next, int32_t* __restrict__ exited, int32_t* __restrict__ exit_layer,
    int max_n) {
  __shared__ int sh[kThreads / 64 + 1];
  const int n = min(*n_active, max_n);
  const int start = blockIdx.x * kTile;
  if (start >= n) return;
  const int end = min(n, start + kTile);
  int ex = tile_ex[blockIdx.x];
  int keep = start - ex;
  split_range(start, end, layer, flags, active, next, exited, exit_layer, &keep, &ex, sh);
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_compact_workspace_bytes(int max_active) {
  if (max_active <= kSingleMax) return 0;
  return (size_t)ceil_div(max_active, kTile) * sizeof(int32_t);
}

extern "C" adept_status adept_compact(int layer, const uint8_t* exit_flag,
                                      const int32_t* active_rows, const int32_t* n_active,
                                      int max_active, int32_t* next_rows, int32_t* n_next,
                                      int32_t* exited_rows, int32_t* n_exited,
                                      int32_t* exit_layer, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  ADEPT_REQUIRE(max_active >= 0, "compact: max_active < 0");
  ADEPT_REQUIRE(exit_flag && active_rows && n_active && next_rows && n_next && exited_rows &&
                    n_exited && exit_layer,
                "compact: NULL tensor");
  ADEPT_REQUIRE(aligned16(active_rows) && ((uintptr_t)exit_flag & 3) == 0,
                "compact: active_rows must be 16-byte and exit_flag 4-byte aligned");
  ADEPT_REQUIRE(next_rows != active_rows && exited_rows != active_rows,
                "compact: outputs must not alias active_rows");
  hipStream_t s = as_stream(stream);
  if (max_active <= kSingleMax) {
    ADEPT_LAUNCH(compact_single, dim3(1), dim3(kThreads), 0, s, layer, exit_flag,
                       active_rows, n_active, next_rows, n_next, exited_rows, n_exited,
                       exit_layer, max_active);
    return launch_status("compact");
  }
  const size_t need = adept_compact_workspace_bytes(max_active);
  if (!workspace || workspace_bytes < need) {
    set_error("compact: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  const int tiles = ceil_div(max_active, kTile);
  int32_t* tile_ex = (int32_t*)workspace;
  ADEPT_LAUNCH(compact_count, dim3(tiles), dim3(kThreads), 0, s, exit_flag, n_active,
                     tile_ex, max_active);
  ADEPT_CHECK_LAUNCH("compact_count");
  ADEPT_LAUNCH(compact_scan, dim3(1), dim3(kThreads), 0, s, n_active, tile_ex, n_next,
                     n_exited, max_active);
  ADEPT_CHECK_LAUNCH("compact_scan");
  ADEPT_LAUNCH(compact_scatter, dim3(tiles), dim3(kThreads), 0, s, layer, exit_flag,
                     active_rows, n_active, tile_ex, next_rows, exited_rows, exit_layer,
                     max_active);
  return launch_status("compact_scatter");
}
