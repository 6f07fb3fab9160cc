// Token-level exit test (Section 4.1, Eq. 7-8; local metric of Appendix H.3).
//
// One wavefront per active row.  Each lane reads 16-byte vectors of the row
// (8 bf16 or 4 f32 values) at vector index c*64 + lane, keeps them in
// registers, and accumulates the three sums <h,h>, <r,r>, <h,r> in double
// (every product of two float values is exact in double).  A xor butterfly
// reduces across the wave; the decision is taken in double.  For the global
// metric the inertia row is then updated from the registers, so each byte
// of h and of the inertia crosses HBM once (read h, read + write inertia).
#include "common.h"

namespace adept {
namespace {

constexpr int kWavesPerBlock = 4;

struct ExitParams {
  double delta;
  int min_exit_layer, n_layers, layer, d;
};

template <typename T> struct Vec16;
template <> struct Vec16<float> { static constexpr int n = 4; };
template <> struct Vec16<bf16> { static constexpr int n = 8; };

// Element i of a 16-byte vector of T, as float.
template <typename T> __device__ __forceinline__ float elem(const uint4& r, int i);
template <> __device__ __forceinline__ float elem<float>(const uint4& r, int i) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
  return __uint_as_float(w[i]);
}
template <> __device__ __forceinline__ float elem<bf16>(const uint4& r, int i) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
  return __uint_as_float((i & 1) ? (w[i >> 1] & 0xffff0000u) : (w[i >> 1] << 16));
}

// Values stay in registers in their stored form (16-byte vectors, bf16
// packed) between the reduction and the inertia update, which keeps the
// register count low enough for several rows in flight per SIMD.
template <typename T, int CH, bool GLOBAL>
__global__ __launch_bounds__(64 * kWavesPerBlock) void exit_test_kernel(
    ExitParams p, int max_active, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_active,
    const T* __restrict__ h_cur, const T* __restrict__ h_prev, float* __restrict__ inertia,
    const int32_t* __restrict__ force_layer, uint8_t* __restrict__ exit_flag,
    double* __restrict__ sim_out) {
  constexpr int V = Vec16<T>::n;
  constexpr int RV = GLOBAL ? V / 4 : 1;   // 16-byte vectors of the reference per chunk
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (k >= min(*n_active, max_active)) return;
  const int row = rows[k];
  const int nvec = p.d / V;
  const T* hr = h_cur + (int64_t)row * p.d;

  uint4 hv[CH];
  uint4 rv[CH][RV];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int vi = c * 64 + lane;
    if (vi < nvec) {
      hv[c] = *reinterpret_cast<const uint4*>(hr + vi * V);
      if (GLOBAL) {
        const float* ir = inertia + (int64_t)row * p.d + vi * V;
#pragma unroll
        for (int q = 0; q < RV; ++q) rv[c][q] = *reinterpret_cast<const uint4*>(ir + 4 * q);
      } else {
        rv[c][0] = *reinterpret_cast<const uint4*>(h_prev + (int64_t)row * p.d + vi * V);
      }
    }
  }
  double s_hh = 0.0, s_rr = 0.0, s_hr = 0.0;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int vi = c * 64 + lane;
    if (vi < nvec) {
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const double a = elem<T>(hv[c], v);
        const double b = GLOBAL ? elem<float>(rv[c][v >> 2], v & 3) : elem<T>(rv[c][0], v);
        s_hh = fma(a, a, s_hh);
        s_rr = fma(b, b, s_rr);
        s_hr = fma(a, b, s_hr);
      }
    }
  }
  s_hh = wave_sum_f64(s_hh);
  s_rr = wave_sum_f64(s_rr);
  s_hr = wave_sum_f64(s_hr);

  const double nh = sqrt(s_hh), nr = sqrt(s_rr);
  const double den = nh * nr;
  const double sim = den > 0.0 ? s_hr / den : __longlong_as_double(0x7ff8000000000000ll);
  bool ex = (p.layer >= p.min_exit_layer) && (p.layer <= p.n_layers - 1) && (sim >= p.delta);
  if (force_layer) {
    const int f = force_layer[row];
    if (f > 0) ex = (p.layer == f) && (p.layer <= p.n_layers - 1);
  }
  if (lane == 0) {
    exit_flag[k] = ex ? 1 : 0;
    if (sim_out) sim_out[k] = sim;
  }
  if (GLOBAL && nh > 0.0) {
    const double inv = 1.0 / nh;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int vi = c * 64 + lane;
      if (vi < nvec) {
        float* ir = inertia + (int64_t)row * p.d + vi * V;
#pragma unroll
        for (int q = 0; q < RV; ++q) {
          float4 o;
          o.x = (float)((double)elem<float>(rv[c][q], 0) + (double)elem<T>(hv[c], 4 * q + 0) * inv);
          o.y = (float)((double)elem<float>(rv[c][q], 1) + (double)elem<T>(hv[c], 4 * q + 1) * inv);
          o.z = (float)((double)elem<float>(rv[c][q], 2) + (double)elem<T>(hv[c], 4 * q + 2) * inv);
          o.w = (float)((double)elem<float>(rv[c][q], 3) + (double)elem<T>(hv[c], 4 * q + 3) * inv);
          *reinterpret_cast<float4*>(ir + 4 * q) = o;
        }
      }
    }
  }
}

template <typename T, bool GLOBAL>
adept_status launch_exit(int ch, const ExitParams& p, int max_active, const int32_t* rows,
                         const int32_t* n_active, const void* h_cur, const void* h_prev,
                         float* inertia, const int32_t* force, uint8_t* flag, double* sim,
                         hipStream_t s) {
  dim3 grid(ceil_div(max_active, kWavesPerBlock)), block(64 * kWavesPerBlock);
  const T* hc = (const T*)h_cur;
  const T* hp = (const T*)h_prev;
#define ADEPT_EXIT_CASE(C)                                                                     \
  case C:                                                                                      \
    ADEPT_LAUNCH((exit_test_kernel<T, C, GLOBAL>), grid, block, 0, s, p, max_active, rows, n_active, \
                       hc, hp, inertia, force, flag, sim);                                     \
    break;
  switch (ch) {
    ADEPT_EXIT_CASE(1)
    ADEPT_EXIT_CASE(2)
    ADEPT_EXIT_CASE(4)
    ADEPT_EXIT_CASE(8)
    default:
      set_error("exit_test: unsupported chunk count %d", ch);
      return ADEPT_E_UNSUPPORTED;
  }
#undef ADEPT_EXIT_CASE
  return launch_status("exit_test");
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" adept_status adept_exit_test(adept_dtype dt, int d_model, int layer,
                                        const adept_exit_cfg* cfg, const int32_t* active_rows,
                                        const int32_t* n_active, int max_active,
                                        const void* h_cur, const void* h_prev, float* inertia,
                                        const int32_t* force_layer, uint8_t* exit_flag,
                                        double* sim_out, void* stream) {
  ADEPT_REQUIRE(cfg != nullptr, "exit_test: cfg is NULL");
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "exit_test: bad dtype %d", (int)dt);
  ADEPT_REQUIRE(cfg->metric == ADEPT_SIM_GLOBAL || cfg->metric == ADEPT_SIM_LOCAL,
                "exit_test: bad metric %d", cfg->metric);
  ADEPT_REQUIRE(cfg->n_layers >= 1 && layer >= 1 && layer <= cfg->n_layers,
                "exit_test: layer %d outside 1..%d", layer, cfg->n_layers);
  ADEPT_REQUIRE(max_active >= 0, "exit_test: max_active < 0");
  ADEPT_REQUIRE(!std::isnan(cfg->delta), "exit_test: delta is NaN");
  const int V = dt == ADEPT_BF16 ? 8 : 4;
  ADEPT_REQUIRE(d_model > 0 && d_model % V == 0, "exit_test: d_model %d not a multiple of %d",
                d_model, V);
  const bool global = cfg->metric == ADEPT_SIM_GLOBAL;
  ADEPT_REQUIRE(active_rows && n_active && h_cur && exit_flag, "exit_test: NULL tensor");
  ADEPT_REQUIRE(global ? inertia != nullptr : h_prev != nullptr,
                "exit_test: %s needs %s", global ? "GLOBAL" : "LOCAL",
                global ? "inertia" : "h_prev");
  ADEPT_REQUIRE(aligned16(h_cur) && (!h_prev || aligned16(h_prev)) &&
                    (!inertia || aligned16(inertia)),
                "exit_test: tensors must be 16-byte aligned");
  if (max_active == 0) return ADEPT_OK;
  const int nvec = d_model / V;
  int ch = (nvec + 63) / 64;
  int chp = 1;
  while (chp < ch) chp <<= 1;
  if (chp > 8) {
    set_error("exit_test: d_model %d too large (max %d)", d_model, 8 * 64 * V);
    return ADEPT_E_UNSUPPORTED;
  }
  ExitParams p{cfg->delta, cfg->min_exit_layer, cfg->n_layers, layer, d_model};
  hipStream_t s = as_stream(stream);
  if (dt == ADEPT_BF16) {
    return global ? launch_exit<bf16, true>(chp, p, max_active, active_rows, n_active, h_cur,
                                            h_prev, inertia, force_layer, exit_flag, sim_out, s)
                  : launch_exit<bf16, false>(chp, p, max_active, active_rows, n_active, h_cur,
                                             h_prev, inertia, force_layer, exit_flag, sim_out, s);
  }
  return global ? launch_exit<float, true>(chp, p, max_active, active_rows, n_active, h_cur,
                                           h_prev, inertia, force_layer, exit_flag, sim_out, s)
                : launch_exit<float, false>(chp, p, max_active, active_rows, n_active, h_cur,
                                            h_prev, inertia, force_layer, exit_flag, sim_out, s);
}
