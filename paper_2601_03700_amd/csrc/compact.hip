// Active-index update of Appendix I: stable split of the active list by the
// exit flags into the rows that continue and the rows that exit.
//
// The split is wave-ballot based.  A workgroup of 16 waves takes a range of
// the list; each wave owns a contiguous chunk of it (a multiple of 64
// entries).  Pass A: per 64 entries the wave takes one 64-bit ballot of the
// exit flags (kept in LDS) and counts exits.  The 16 wave totals are scanned
// in LDS.  Pass B: lane l of a 64-entry step reads its row (coalesced) and
// writes it at (wave offset + popcount of the ballot below l) among the exits
// or at (wave offset + l - that count) among the kept rows, so stores of a
// wave land on consecutive addresses.  Lists up to 64K entries (the
// per-layer case) use one workgroup over the whole list; longer lists use
// three passes over 16K-entry tiles: a count of exits per tile (16 flags per
// thread, one 16-byte load), a scan of the tile counts, and the split of
// each tile from its offsets.  Input order is kept in both outputs.
#include "common.h"

namespace adept {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kTileItems = 16;                 // flags per thread in the count pass
constexpr int kTile = kThreads * kTileItems;   // multi-pass tile = 16K entries
constexpr int kSingleMax = 1 << 16;            // lists up to this use one workgroup
constexpr int kMaxSteps = kSingleMax / kThreads;   // 64-entry steps per wave, at most
constexpr int kBatch = 16;                     // steps whose loads are issued together

// Splits entries [start, end) with the block's waves on consecutive chunks of
// `chunk` entries (a multiple of 64, chunk * kWaves >= end - start).  Exits go
// to exited[ex_base + ...], kept rows to next[keep_base + ...].  Steps are
// taken kBatch at a time so that a batch's loads are in flight together.
__device__ __forceinline__ void split_block(int start, int end, int chunk, int ex_base,
                                            int keep_base, int layer,
                                            const uint8_t* __restrict__ flags,
                                            const int32_t* __restrict__ active,
                                            int32_t* __restrict__ next,
                                            int32_t* __restrict__ exited,
                                            int32_t* __restrict__ exit_layer, uint64_t* masks,
                                            int* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lo = start + wave * chunk;
  const int hi = min(end, lo + chunk);
  const int steps = chunk >> 6;
  uint64_t* wm = masks + wave * steps;
  int ex = 0;
  for (int s0 = 0; s0 < steps; s0 += kBatch) {
    uint8_t f[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int e = lo + (s0 + b) * 64 + lane;
      f[b] = (s0 + b < steps && e < hi) ? flags[e] : 0;
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      if (s0 + b < steps) {
        const uint64_t m = __ballot(f[b] != 0);
        if (lane == 0) wm[s0 + b] = m;
        ex += __popcll(m);
      }
    }
  }
  if (lane == 0) {
    sh[wave] = ex;
    sh[kWaves + wave] = max(0, hi - lo) - ex;
  }
  __syncthreads();
  int ex_off = ex_base, keep_off = keep_base;
  for (int w = 0; w < wave; ++w) {
    ex_off += sh[w];
    keep_off += sh[kWaves + w];
  }
  const uint64_t lt = (1ull << lane) - 1ull;   // lanes below this one
  for (int s0 = 0; s0 < steps && lo + s0 * 64 < hi; s0 += kBatch) {
    int32_t r[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int e = lo + (s0 + b) * 64 + lane;
      r[b] = (s0 + b < steps && e < hi) ? active[e] : 0;
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int base = lo + (s0 + b) * 64;
      if (s0 + b < steps && base < hi) {
        const uint64_t m = wm[s0 + b];
        if (base + lane < hi) {
          const int below = __popcll(m & lt);
          if ((m >> lane) & 1ull) {
            exited[ex_off + below] = r[b];
            exit_layer[r[b]] = layer;
          } else {
            next[keep_off + lane - below] = r[b];
          }
        }
        const int me = __popcll(m);
        ex_off += me;
        keep_off += min(64, hi - base) - me;
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void compact_single(
    int layer, const uint8_t* __restrict__ flags, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active, int32_t* __restrict__ next, int32_t* __restrict__ n_next,
    int32_t* __restrict__ exited, int32_t* __restrict__ n_exited,
    int32_t* __restrict__ exit_layer, int max_n) {
  __shared__ uint64_t masks[kWaves * kMaxSteps];
  __shared__ int sh[2 * kWaves];
  const int n = min(*n_active, max_n);     // max_n <= kSingleMax
  const int chunk = ((n + kThreads - 1) / kThreads) * 64;   // ceil(n / kWaves) rounded to 64
  split_block(0, n, chunk, 0, 0, layer, flags, active, next, exited, exit_layer, masks, sh);
  if (threadIdx.x == 0) {
    int ex = 0;
    for (int w = 0; w < kWaves; ++w) ex += sh[w];
    *n_exited = ex;
    *n_next = n - ex;
  }
}

// Inclusive scan of v over the workgroup; returns the exclusive prefix and
// writes the workgroup total to *total.  `sh` holds >= kWaves + 1 ints.
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
    for (int w = 0; w < kWaves; ++w) {
      const int t = sh[w];
      sh[w] = run;
      run += t;
    }
    sh[kWaves] = run;
  }
  __syncthreads();
  const int excl = sh[wave] + x - v;
  *total = sh[kWaves];
  __syncthreads();
  return excl;
}

// pass 1: exits per tile
__global__ __launch_bounds__(kThreads) void compact_count(const uint8_t* __restrict__ flags,
                                                          const int32_t* __restrict__ n_active,
                                                          int32_t* __restrict__ tile_ex,
                                                          int max_n) {
  __shared__ int sh[kWaves + 1];
  const int n = min(*n_active, max_n);
  const int start = blockIdx.x * kTile;
  if (start >= n) return;
  const int end = min(n, start + kTile);
  // kTileItems flags per thread: one 16-byte load, nonzero bytes counted
  static_assert(kTileItems == 16, "one uint4 of flags per thread");
  const int e0 = start + threadIdx.x * kTileItems;
  int cnt = 0;
  if (e0 + kTileItems <= end) {
    const uint4 v = *reinterpret_cast<const uint4*>(flags + e0);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t x = w[q];
      x |= x >> 4;
      x |= x >> 2;
      x |= x >> 1;
      cnt += __popc(x & 0x01010101u);
    }
  } else {
    for (int e = e0; e < end && e < e0 + kTileItems; ++e) cnt += flags[e] ? 1 : 0;
  }
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
  __shared__ int sh[kWaves + 1];
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

// pass 3: split each tile from its offsets
__global__ __launch_bounds__(kThreads) void compact_scatter(
    int layer, const uint8_t* __restrict__ flags, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active, const int32_t* __restrict__ tile_ex,
    int32_t* __restrict__ next, int32_t* __restrict__ exited, int32_t* __restrict__ exit_layer,
    int max_n) {
  __shared__ uint64_t masks[kTile / 64];
  __shared__ int sh[2 * kWaves];
  const int n = min(*n_active, max_n);
  const int start = blockIdx.x * kTile;
  if (start >= n) return;
  const int end = min(n, start + kTile);
  const int ex = tile_ex[blockIdx.x];
  split_block(start, end, kTile / kWaves, ex, start - ex, layer, flags, active, next, exited,
              exit_layer, masks, sh);
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
  ADEPT_REQUIRE(aligned16(exit_flag),
                "compact: exit_flag must be 16-byte aligned above %d entries", kSingleMax);
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
