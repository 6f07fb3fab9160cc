// Token-level exit test (Section 4.1, Eq. 7-8; local metric of Appendix H.3).
//
// One wavefront per active row.  Per chunk c each lane holds E consecutive
// elements of h starting at element (c*64 + lane)*E, with E = 4 for the
// global metric (8 bytes of bf16 h beside one contiguous 16-byte vector of
// the f32 inertia) and E = 16/sizeof(T) for the local one, so that every
// load and store instruction of the wave covers one contiguous span.  The
// values stay in registers in their stored form between the reduction and
// the inertia update; the three sums <h,h>, <r,r>, <h,r> are accumulated in
// double (every product of two float values is exact in double), a xor
// butterfly reduces across the wave and the decision is taken in double.
// For the global metric the inertia row is then updated from the registers,
// so each byte of h and of the inertia crosses HBM once (read h, read +
// write inertia).  Every access is streaming (non-temporal): nothing the
// kernel touches is read again before it has left the caches.  The combined
// metric (both cosines must reach the threshold) reads h, h_prev and the
// inertia with the global metric's grouping (4 elements per lane and chunk)
// and keeps five sums.
#include "common.h"

namespace adept {
namespace {

constexpr int kWavesPerBlock = 4;
constexpr int kMaxChunks = 32;
constexpr int kMaxChunksBoth = 16;   // three row streams in registers

enum Mode { kLocal = 0, kGlobal = 1, kBoth = 2 };

struct ExitParams {
  double delta;
  int min_exit_layer, n_layers, layer, d;
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <int BYTES> struct Raw;
template <> struct Raw<8> { using type = u32x2; };
template <> struct Raw<16> { using type = u32x4; };

// Element i of a raw vector of T, as float.
template <typename T, typename R> __device__ __forceinline__ float elem(const R& r, int i) {
  if constexpr (sizeof(T) == 4) {
    return __uint_as_float(r[i]);
  } else {
    const uint32_t w = r[i >> 1];
    return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
  }
}

template <typename T, int CH, int MODE>
__global__ __launch_bounds__(64 * kWavesPerBlock)
void exit_test_kernel(
    ExitParams p, int max_active, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_active,
    const T* __restrict__ h_cur, const T* __restrict__ h_prev, float* __restrict__ inertia,
    const int32_t* __restrict__ force_layer, uint8_t* __restrict__ exit_flag,
    double* __restrict__ sim_out) {
  constexpr bool GLOBAL = MODE != kLocal;   // reads and updates the inertia
  constexpr bool BOTH = MODE == kBoth;      // also reads h_prev
  constexpr int E = GLOBAL ? 4 : 16 / (int)sizeof(T);
  using HRaw = typename Raw<E * sizeof(T)>::type;
  using RRaw = u32x4;   // 4 f32 of the inertia, or E values of h_prev
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (k >= min(*n_active, max_active)) return;
  const int row = rows[k];
  const int nvec = p.d / E;
  const T* hr = h_cur + (int64_t)row * p.d;
  const uint32_t* rr = GLOBAL ? reinterpret_cast<const uint32_t*>(inertia + (int64_t)row * p.d)
                              : reinterpret_cast<const uint32_t*>(h_prev + (int64_t)row * p.d);

  const T* pr = BOTH ? h_prev + (int64_t)row * p.d : nullptr;   // combined metric only

  HRaw hv[CH];
  RRaw rv[CH];
  HRaw pv[BOTH ? CH : 1];
  // Loads are not predicated: a lane past the end of the row re-reads the
  // row's last vector and contributes zeros (predicated loads leave the
  // register allocator with partially defined values and cost spills).
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int vi = min(c * 64 + lane, nvec - 1);
    hv[c] = __builtin_nontemporal_load(reinterpret_cast<const HRaw*>(hr + vi * E));
    rv[c] = __builtin_nontemporal_load(reinterpret_cast<const RRaw*>(rr) + vi);
    if constexpr (BOTH) pv[c] = __builtin_nontemporal_load(reinterpret_cast<const HRaw*>(pr + vi * E));
  }
  double s_hh = 0.0, s_rr = 0.0, s_hr = 0.0, s_pp = 0.0, s_hp = 0.0;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const bool live = c * 64 + lane < nvec;
#pragma unroll
    for (int v = 0; v < E; ++v) {
      const double a = live ? elem<T>(hv[c], v) : 0.0f;
      const double b = live ? (GLOBAL ? elem<float>(rv[c], v) : elem<T>(rv[c], v)) : 0.0f;
      s_hh = fma(a, a, s_hh);
      s_rr = fma(b, b, s_rr);
      s_hr = fma(a, b, s_hr);
      if constexpr (BOTH) {
        const double q = live ? elem<T>(pv[c], v) : 0.0f;
        s_pp = fma(q, q, s_pp);
        s_hp = fma(a, q, s_hp);
      }
    }
    // chunk by chunk: the conversions to double are not hoisted (and held
    // in registers) ahead of the chunk that needs them
    __builtin_amdgcn_sched_barrier(0);
  }
  s_hh = wave_sum_f64(s_hh);
  s_rr = wave_sum_f64(s_rr);
  s_hr = wave_sum_f64(s_hr);
  if constexpr (BOTH) {
    s_pp = wave_sum_f64(s_pp);
    s_hp = wave_sum_f64(s_hp);
  }

  const double kNaN = __longlong_as_double(0x7ff8000000000000ll);
  const double nh = sqrt(s_hh), nr = sqrt(s_rr);
  const double den = nh * nr;
  double sim = den > 0.0 ? s_hr / den : kNaN;
  bool pass = sim >= p.delta;
  if constexpr (BOTH) {
    // the local cosine must pass too; the reported similarity is the
    // smaller of the two (NaN if either is undefined)
    const double den_l = nh * sqrt(s_pp);
    const double sim_l = den_l > 0.0 ? s_hp / den_l : kNaN;
    pass = pass && sim_l >= p.delta;
    sim = (sim != sim || sim_l != sim_l) ? kNaN : fmin(sim, sim_l);
  }
  const bool ex = exit_decision(pass, p.layer, p.min_exit_layer, p.n_layers, force_layer, row);
  if (lane == 0) {
    exit_flag[k] = ex ? 1 : 0;
    if (sim_out) sim_out[k] = sim;
  }
  if (GLOBAL && nh > 0.0) {
    const double inv = 1.0 / nh;
    float* iw = inertia + (int64_t)row * p.d;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      // opaque to the optimiser: the values are converted again here rather
      // than kept in double registers since the reduction
      asm volatile("" : "+v"(hv[c]), "+v"(rv[c]));
      const int vi = c * 64 + lane;
      if (vi < nvec) {
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          o[e] = __float_as_uint(
              (float)((double)elem<float>(rv[c], e) + (double)elem<T>(hv[c], e) * inv));
        __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(iw) + vi);
      }
    }
  }
}

template <typename T, int MODE>
adept_status launch_exit(int ch, const ExitParams& p, int max_active, const int32_t* rows,
                         const int32_t* n_active, const void* h_cur, const void* h_prev,
                         float* inertia, const int32_t* force, uint8_t* flag, double* sim,
                         hipStream_t s) {
  dim3 grid(ceil_div(max_active, kWavesPerBlock)), block(64 * kWavesPerBlock);
  const T* hc = (const T*)h_cur;
  const T* hp = (const T*)h_prev;
#define ADEPT_EXIT_CASE(C)                                                                     \
  case C:                                                                                      \
    ADEPT_LAUNCH((exit_test_kernel<T, C, MODE>), grid, block, 0, s, p, max_active, rows, n_active, \
                       hc, hp, inertia, force, flag, sim);                                     \
    break;
  switch (MODE == kBoth && ch > kMaxChunksBoth ? 0 : ch) {
    ADEPT_EXIT_CASE(1)
    ADEPT_EXIT_CASE(2)
    ADEPT_EXIT_CASE(4)
    ADEPT_EXIT_CASE(8)
    ADEPT_EXIT_CASE(16)
    case 32:
      if constexpr (MODE != kBoth) {
        ADEPT_LAUNCH((exit_test_kernel<T, 32, MODE>), grid, block, 0, s, p, max_active, rows,
                     n_active, hc, hp, inertia, force, flag, sim);
        break;
      }
      [[fallthrough]];
    default:
      set_error("exit_test: unsupported chunk count %d", ch);
      return ADEPT_E_UNSUPPORTED;
  }
#undef ADEPT_EXIT_CASE
  return launch_status("exit_test");
}

// All-at-once variant (Appendix H.2).  Key of an active row: (position + 1)
// in the high word, its list index in the low word; the largest key of a
// sequence names its last prompt token.
__global__ __launch_bounds__(256) void prompt_level_clear(unsigned long long* __restrict__ key,
                                                          int n_seq) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b < n_seq) key[b] = 0ull;
}

__global__ __launch_bounds__(256) void prompt_level_pick(
    const int32_t* __restrict__ rows, const int32_t* __restrict__ n_active, int max_active,
    const int32_t* __restrict__ seq, const int32_t* __restrict__ pos, int n_seq,
    unsigned long long* __restrict__ key) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= min(*n_active, max_active)) return;
  const int row = rows[k];
  const int b = seq[row];
  if (b < 0 || b >= n_seq) return;
  atomicMax(&key[b], ((unsigned long long)(uint32_t)(pos[row] + 1) << 32) | (uint32_t)k);
}

__global__ __launch_bounds__(256) void prompt_level_apply(
    const int32_t* __restrict__ rows, const int32_t* __restrict__ n_active, int max_active,
    const int32_t* __restrict__ seq, int n_seq, const unsigned long long* __restrict__ key,
    uint8_t* flag) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= min(*n_active, max_active)) return;
  const int b = seq[rows[k]];
  if (b < 0 || b >= n_seq) return;
  // the deciding row rewrites its own flag with the value it already holds
  flag[k] = flag[(uint32_t)key[b]];
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_exit_prompt_level_workspace_bytes(int n_seq) {
  return n_seq > 0 ? (size_t)n_seq * sizeof(unsigned long long) : 0;
}

extern "C" adept_status adept_exit_prompt_level(const int32_t* active_rows,
                                                const int32_t* n_active, int max_active,
                                                const int32_t* seq, const int32_t* pos, int n_seq,
                                                uint8_t* exit_flag, void* workspace,
                                                size_t workspace_bytes, void* stream) {
  ADEPT_REQUIRE(max_active >= 0 && n_seq >= 0, "exit_prompt_level: negative size");
  ADEPT_REQUIRE(active_rows && n_active && seq && pos && exit_flag,
                "exit_prompt_level: NULL tensor");
  if (max_active == 0 || n_seq == 0) return ADEPT_OK;
  const size_t need = adept_exit_prompt_level_workspace_bytes(n_seq);
  if (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 7)) {
    set_error("exit_prompt_level: workspace of %zu bytes (8-byte aligned) needed", need);
    return ADEPT_E_WORKSPACE;
  }
  hipStream_t s = as_stream(stream);
  auto* key = (unsigned long long*)workspace;
  ADEPT_LAUNCH(prompt_level_clear, dim3(ceil_div(n_seq, 256)), dim3(256), 0, s, key, n_seq);
  ADEPT_CHECK_LAUNCH("prompt_level_clear");
  ADEPT_LAUNCH(prompt_level_pick, dim3(ceil_div(max_active, 256)), dim3(256), 0, s, active_rows,
               n_active, max_active, seq, pos, n_seq, key);
  ADEPT_CHECK_LAUNCH("prompt_level_pick");
  ADEPT_LAUNCH(prompt_level_apply, dim3(ceil_div(max_active, 256)), dim3(256), 0, s, active_rows,
               n_active, max_active, seq, n_seq, key, exit_flag);
  return launch_status("prompt_level_apply");
}

extern "C" adept_status adept_exit_test(adept_dtype dt, int d_model, int layer,
                                        const adept_exit_cfg* cfg, const int32_t* active_rows,
                                        const int32_t* n_active, int max_active,
                                        const void* h_cur, const void* h_prev, float* inertia,
                                        const int32_t* force_layer, uint8_t* exit_flag,
                                        double* sim_out, void* stream) {
  ADEPT_REQUIRE(cfg != nullptr, "exit_test: cfg is NULL");
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "exit_test: bad dtype %d", (int)dt);
  ADEPT_REQUIRE(cfg->metric == ADEPT_SIM_GLOBAL || cfg->metric == ADEPT_SIM_LOCAL ||
                    cfg->metric == ADEPT_SIM_BOTH,
                "exit_test: bad metric %d", cfg->metric);
  ADEPT_REQUIRE(cfg->n_layers >= 1 && layer >= 1 && layer <= cfg->n_layers,
                "exit_test: layer %d outside 1..%d", layer, cfg->n_layers);
  ADEPT_REQUIRE(max_active >= 0, "exit_test: max_active < 0");
  ADEPT_REQUIRE(!std::isnan(cfg->delta), "exit_test: delta is NaN");
  ADEPT_REQUIRE(cfg->prompt_level == 0 || cfg->prompt_level == 1,
                "exit_test: prompt_level %d is not 0 or 1", cfg->prompt_level);
  const bool global = cfg->metric != ADEPT_SIM_LOCAL;   // GLOBAL or BOTH: inertia
  const bool both = cfg->metric == ADEPT_SIM_BOTH;
  // elements per lane and chunk (kernel's E)
  const int V = global ? 4 : (dt == ADEPT_BF16 ? 8 : 4);
  ADEPT_REQUIRE(d_model > 0 && d_model % V == 0, "exit_test: d_model %d not a multiple of %d",
                d_model, V);
  ADEPT_REQUIRE(active_rows && n_active && h_cur && exit_flag, "exit_test: NULL tensor");
  ADEPT_REQUIRE(!global || inertia != nullptr, "exit_test: GLOBAL/BOTH need inertia");
  ADEPT_REQUIRE((global && !both) || h_prev != nullptr, "exit_test: LOCAL/BOTH need h_prev");
  ADEPT_REQUIRE(aligned16(h_cur) && (!h_prev || aligned16(h_prev)) &&
                    (!inertia || aligned16(inertia)),
                "exit_test: tensors must be 16-byte aligned");
  if (max_active == 0) return ADEPT_OK;
  const int nvec = d_model / V;
  int ch = (nvec + 63) / 64;
  int chp = 1;
  while (chp < ch) chp <<= 1;
  const int max_ch = both ? kMaxChunksBoth : kMaxChunks;
  if (chp > max_ch) {
    set_error("exit_test: d_model %d too large (max %d)", d_model, max_ch * 64 * V);
    return ADEPT_E_UNSUPPORTED;
  }
  ExitParams p{cfg->delta, cfg->min_exit_layer, cfg->n_layers, layer, d_model};
  hipStream_t s = as_stream(stream);
#define ADEPT_EXIT_MODE(T)                                                                   \
  switch (cfg->metric) {                                                                     \
    case ADEPT_SIM_GLOBAL:                                                                   \
      return launch_exit<T, kGlobal>(chp, p, max_active, active_rows, n_active, h_cur, h_prev, \
                                     inertia, force_layer, exit_flag, sim_out, s);           \
    case ADEPT_SIM_LOCAL:                                                                    \
      return launch_exit<T, kLocal>(chp, p, max_active, active_rows, n_active, h_cur, h_prev,  \
                                    inertia, force_layer, exit_flag, sim_out, s);            \
    default:                                                                                 \
      return launch_exit<T, kBoth>(chp, p, max_active, active_rows, n_active, h_cur, h_prev,   \
                                   inertia, force_layer, exit_flag, sim_out, s);             \
  }
  if (dt == ADEPT_BF16) {
    ADEPT_EXIT_MODE(bf16)
  }
  ADEPT_EXIT_MODE(float)
#undef ADEPT_EXIT_MODE
}
