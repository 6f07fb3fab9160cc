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
// 16-byte load, four loads per thread) that also stores the 64-bit exit mask
// of every 64 entries, a scan of the tile counts, and the split of each tile from its
// offsets, which reads the masks (one bit per entry) instead of the flags.
// Input order is kept in both outputs.
#include "common.h"

namespace adept {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kTile = 1 << 14;                 // multi-pass tile = 16K entries
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

// pass 1: exits per tile.  256 threads per 16K-entry tile; thread t reads
// the 16 flags at 16 * (j * 256 + t) for j < 4 (four 16-byte loads in
// flight, each instruction of a wave on 1 KB of consecutive flags).  The four
// threads of a quad then hold 64 consecutive entries, whose exit bits the
// quad's first thread stores as one 64-bit mask.
constexpr int kCountThreads = 256;
constexpr int kCountLoads = kTile / (kCountThreads * 16);   // 4
__global__ __launch_bounds__(kCountThreads) void compact_count(
    const uint8_t* __restrict__ flags, const int32_t* __restrict__ n_active,
    int32_t* __restrict__ tile_ex, uint64_t* __restrict__ masks, int max_n) {
  __shared__ int sh[kCountThreads / 64];
  const int n = min(*n_active, max_n);
  const int start = blockIdx.x * kTile;
  if (start >= n) return;
  const int end = min(n, start + kTile);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 v[kCountLoads];
#pragma unroll
  for (int j = 0; j < kCountLoads; ++j) {
    const int e0 = start + (j * kCountThreads + (int)threadIdx.x) * 16;
    // the load is clamped to the array's last whole 16 bytes and its value
    // used only when all 16 flags lie before `end`
    const int ec = min(e0, (max_n - 16) & ~15);
    v[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(flags + ec));
    if (e0 + 16 > end) v[j] = u32x4{0u, 0u, 0u, 0u};
  }
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < kCountLoads; ++j) {
    const int e0 = start + (j * kCountThreads + (int)threadIdx.x) * 16;
    uint32_t m16 = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
        if ((v[j][q] >> (8 * bb)) & 0xffu) m16 |= 1u << (4 * q + bb);
    if (e0 < end && e0 + 16 > end) {   // the row's ragged end: byte loads
      for (int e = e0; e < end; ++e)
        if (flags[e]) m16 |= 1u << (e - e0);
    }
    cnt += __popc(m16);
    const uint32_t m1 = __shfl_down(m16, 1, 64), m2 = __shfl_down(m16, 2, 64),
                   m3 = __shfl_down(m16, 3, 64);
    if ((lane & 3) == 0 && e0 < end)
      masks[e0 >> 6] = (uint64_t)m16 | ((uint64_t)m1 << 16) | ((uint64_t)m2 << 32) |
                       ((uint64_t)m3 << 48);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (lane == 0) sh[wave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < kCountThreads / 64; ++w) t += sh[w];
    tile_ex[blockIdx.x] = t;
  }
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

// pass 3: split each tile from its offsets.  The waves own consecutive
// chunks of 1024 entries; a wave reads its 16 exit masks (128 consecutive
// bytes, one bit per entry) instead of the flags, so a lane's output slot is
// a popcount of the lower lanes' bits, and the row loads of all 16 of its
// 64-entry steps are in flight together.  Each step is one store per lane,
// to the exit list or to the kept list, and the exit layer of the exits.
__global__ __launch_bounds__(kThreads) void compact_scatter(
    int layer, int n_layers, const uint64_t* __restrict__ masks, const int32_t* __restrict__ active,
    const int32_t* __restrict__ n_active, const int32_t* __restrict__ tile_ex,
    int32_t* __restrict__ next, int32_t* __restrict__ exited, int32_t* __restrict__ exit_layer,
    int max_n) {
  constexpr int kChunk = kTile / kWaves;      // 1024 entries, 16 steps
  constexpr int kSteps = kChunk / 64;
  __shared__ int sh[2 * kWaves];
  const int n = min(*n_active, max_n);
  const int start = blockIdx.x * kTile;
  if (start >= n) return;
  const int end = min(n, start + kTile);
  const int tex = tile_ex[blockIdx.x];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lo = start + wave * kChunk;
  const int hi = min(end, lo + kChunk);
  // the mask array holds whole tiles (kTile / 64 masks each), so all 16
  // loads stay inside it; masks of steps at or past `hi` are not used
  const uint64_t* wm = masks + (lo >> 6);
  uint64_t m[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) m[st] = wm[st];
  int32_t r[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int e = min(lo + st * 64 + lane, n - 1);   // clamped: in bounds, unused past hi
    r[st] = __builtin_nontemporal_load(active + e);
  }
  int ex = 0;
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    m[st] = lo + st * 64 < hi ? m[st] : 0ull;
    ex += __popcll(m[st]);
  }
  if (lane == 0) {
    sh[wave] = ex;
    sh[kWaves + wave] = max(0, hi - lo) - ex;
  }
  __syncthreads();
  int ex_off = tex, keep_off = start - tex;
  for (int w = 0; w < wave; ++w) {
    ex_off += sh[w];
    keep_off += sh[kWaves + w];
  }
  const uint64_t lt = (1ull << lane) - 1ull;   // lanes below this one
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int base = lo + st * 64;
    const uint64_t mm = m[st];
    const int below = __popcll(mm & lt);
    const bool gone = (mm >> lane) & 1ull;
    int32_t* dst = gone ? exited + (ex_off + below) : next + (keep_off + lane - below);
    // A step whose 64 entries all go to one list stores one contiguous run
    // (non-temporal: whole lines, streamed); a mixed step stores two shorter
    // runs through the cache, which merges the neighbouring steps' pieces of
    // a line before it reaches HBM.  A step of 64 consecutive rows (a dense
    // stretch of the list) with exits writes the exit layers of all of them,
    // n_layers for the rows that continue (the value they hold), so its
    // 256 bytes go out as whole lines instead of a partial-line scatter.
    const bool one_list = mm == 0ull || mm == ~0ull;                // wave-uniform
    const int r0 = __builtin_amdgcn_readfirstlane(r[st]);
    const bool dense = mm != 0ull && base + 64 <= hi && __ballot(r[st] == r0 + lane) == ~0ull;
    if (base + lane < hi) {
      if (one_list)
        __builtin_nontemporal_store(r[st], dst);
      else
        *dst = r[st];
      if (dense)
        __builtin_nontemporal_store(gone ? layer : n_layers, exit_layer + r[st]);
      else if (gone)
        exit_layer[r[st]] = layer;
    }
    const int me = __popcll(mm);
    ex_off += me;
    keep_off += max(0, min(64, hi - base)) - me;
  }
}

}  // namespace
}  // namespace adept
using namespace adept;

extern "C" size_t adept_compact_workspace_bytes(int max_active) {
  if (max_active <= kSingleMax) return 0;
  // tile offsets, then one 64-bit exit mask per 64 entries of every tile
  // (whole tiles, 256-byte aligned)
  const size_t tiles = (size_t)ceil_div(max_active, kTile);
  return ((tiles * sizeof(int32_t) + 255) & ~size_t(255)) + tiles * (kTile / 64) * sizeof(uint64_t);
}

extern "C" adept_status adept_compact(int layer, int n_layers, const uint8_t* exit_flag,
                                      const int32_t* active_rows, const int32_t* n_active,
                                      int max_active, int32_t* next_rows, int32_t* n_next,
                                      int32_t* exited_rows, int32_t* n_exited,
                                      int32_t* exit_layer, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  ADEPT_REQUIRE(max_active >= 0, "compact: max_active < 0");
  ADEPT_REQUIRE(layer >= 1 && layer <= n_layers, "compact: layer %d outside 1..%d", layer, n_layers);
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
  ADEPT_REQUIRE(((uintptr_t)workspace & 7) == 0, "compact: workspace must be 8-byte aligned");
  if (!workspace || workspace_bytes < need) {
    set_error("compact: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  const int tiles = ceil_div(max_active, kTile);
  int32_t* tile_ex = (int32_t*)workspace;
  uint64_t* masks =
      (uint64_t*)((char*)workspace + (((size_t)tiles * sizeof(int32_t) + 255) & ~size_t(255)));
  ADEPT_LAUNCH(compact_count, dim3(tiles), dim3(kCountThreads), 0, s, exit_flag, n_active,
                     tile_ex, masks, max_active);
  ADEPT_CHECK_LAUNCH("compact_count");
  ADEPT_LAUNCH(compact_scan, dim3(1), dim3(kThreads), 0, s, n_active, tile_ex, n_next,
                     n_exited, max_active);
  ADEPT_CHECK_LAUNCH("compact_scan");
  ADEPT_LAUNCH(compact_scatter, dim3(tiles), dim3(kThreads), 0, s, layer, n_layers, masks,
                     active_rows, n_active, tile_ex, next_rows, exited_rows, exit_layer,
                     max_active);
  return launch_status("compact_scatter");
}
