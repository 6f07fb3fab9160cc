// Internal helpers shared by the HIP sources of libadept (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <climits>
#include <stdint.h>

#include <cmath>
#include <cstdio>
#include <string>

#include "../../include/adept.h"

namespace adept {

// ---------------------------------------------------------------------------
// bfloat16 storage (uint16 bit patterns) <-> float
// ---------------------------------------------------------------------------
typedef uint16_t bf16;

__device__ __forceinline__ float bf2f(bf16 x) { return __uint_as_float(((uint32_t)x) << 16); }

// float -> bf16 bits: round to nearest, ties to even; NaN stays a quiet NaN
// (v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ bf16 f2bf(float f) { return __builtin_bit_cast(bf16, (__bf16)f); }
// two floats to a packed pair of bf16 (round to nearest even), a in the low half
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 nbf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, nbf16x2));
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16> {
  __device__ __forceinline__ static float load(const bf16* p) { return bf2f(*p); }
  __device__ __forceinline__ static void store(bf16* p, float v) { *p = f2bf(v); }
};
template <typename T> __device__ __forceinline__ float ld(const T* p) { return Elem<T>::load(p); }
template <typename T> __device__ __forceinline__ void st(T* p, float v) { Elem<T>::store(p, v); }

// MFMA operand / accumulator vector types.
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint16_t)))) uint16_t bf16x4_t;   // 4 bf16 bit patterns
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// ---------------------------------------------------------------------------
// wavefront (64 lanes) reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// The exit decision of Eq. 8 for one row: the test passed (the cosine
// reached delta), inside the window min_exit_layer <= layer <= n_layers - 1;
// a forced schedule (force_layer[row] > 0) overrides it with "exit exactly at
// that layer".
__device__ __forceinline__ bool exit_decision(bool pass, int layer, int min_exit_layer,
                                              int n_layers, const int32_t* force_layer, int row) {
  bool ex = (layer >= min_exit_layer) && (layer <= n_layers - 1) && pass;
  if (force_layer) {
    const int f = force_layer[row];
    if (f > 0) ex = (layer == f) && (layer <= n_layers - 1);
  }
  return ex;
}

// LayerNorm of one bf16 row by one wave, the row held in registers: lane l
// holds the 8-element chunks l, l+64, ..., (R of them; d a multiple of 8 up to
// 512 R, rows 16-byte aligned), so the row crosses HBM once each way and every
// access is a 16-byte vector.  Mean and variance in f32 from the registers
// (two passes); o = (x - mean) / sqrt(var + eps) [* gain + bias].  o may be x.
template <int R>
__device__ __forceinline__ void layernorm_row_vec(const bf16* x, int d, float eps,
                                                  const bf16* __restrict__ gain,
                                                  const bf16* __restrict__ bias, bf16* o,
                                                  int lane) {
  float v[R][8];
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int c = (lane + 64 * j) * 8;
    uint4 w = make_uint4(0, 0, 0, 0);
    if (c < d) w = *reinterpret_cast<const uint4*>(x + c);
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[j][2 * e] = __uint_as_float(u[e] << 16);
      v[j][2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
      s += v[j][2 * e] + v[j][2 * e + 1];
    }
  }
  const float mean = wave_sum_f32(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    if ((lane + 64 * j) * 8 >= d) continue;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float t = v[j][e] - mean;
      q = fmaf(t, t, q);
    }
  }
  const float r = 1.0f / sqrtf(wave_sum_f32(q) / (float)d + eps);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int c = (lane + 64 * j) * 8;
    if (c >= d) continue;
    float y[8];
    if (gain) {
      const uint4 gw = *reinterpret_cast<const uint4*>(gain + c);
      const uint4 bw = *reinterpret_cast<const uint4*>(bias + c);
      const uint32_t gu[4] = {gw.x, gw.y, gw.z, gw.w}, bu[4] = {bw.x, bw.y, bw.z, bw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y[2 * e] = fmaf((v[j][2 * e] - mean) * r, __uint_as_float(gu[e] << 16),
                        __uint_as_float(bu[e] << 16));
        y[2 * e + 1] = fmaf((v[j][2 * e + 1] - mean) * r, __uint_as_float(gu[e] & 0xffff0000u),
                            __uint_as_float(bu[e] & 0xffff0000u));
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * r;
    }
    *reinterpret_cast<uint4*>(o + c) = make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]),
                                                  pack_bf16x2(y[4], y[5]), pack_bf16x2(y[6], y[7]));
  }
}

// 1/sqrt(mean(x^2) + eps) of one row of d elements, by one wave (every lane
// returns it): squares summed in f32 lane by lane (16-byte loads when the row
// allows, several in flight), then across the wave.
template <typename T>
__device__ __forceinline__ float row_rinv_wave(const T* __restrict__ xr, int d, float eps,
                                               int lane) {
  float ss = 0.0f;
  constexpr int V = 16 / sizeof(T);   // elements per 16-byte load
  if (d % V == 0 && ((uintptr_t)xr & 15) == 0) {
#pragma unroll 4
    for (int c = lane * V; c < d; c += 64 * V) {
      const uint4 w = *reinterpret_cast<const uint4*>(xr + c);
      const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if constexpr (sizeof(T) == 2) {
          const float lo = __uint_as_float(u[e] << 16), hi = __uint_as_float(u[e] & 0xffff0000u);
          ss = fmaf(lo, lo, ss);
          ss = fmaf(hi, hi, ss);
        } else {
          const float v = __uint_as_float(u[e]);
          ss = fmaf(v, v, ss);
        }
      }
    }
  } else {
    for (int c = lane; c < d; c += 64) {
      const float v = ld(xr + c);
      ss = fmaf(v, v, ss);
    }
  }
  ss = wave_sum_f32(ss);
  return 1.0f / sqrtf(ss / (float)d + eps);
}

// ---------------------------------------------------------------------------
// host-side error plumbing
// ---------------------------------------------------------------------------
void set_error(const char* fmt, ...);
adept_status launch_status(const char* what);

#define ADEPT_REQUIRE(cond, ...)            \
  do {                                      \
    if (!(cond)) {                          \
      ::adept::set_error(__VA_ARGS__);      \
      return ADEPT_E_INVALID;               \
    }                                       \
  } while (0)

#define ADEPT_CHECK_LAUNCH(what)                                   \
  do {                                                             \
    adept_status _s = ::adept::launch_status(what);                \
    if (_s != ADEPT_OK) return _s;                                 \
  } while (0)

#define ADEPT_TRY(expr)                       \
  do {                                        \
    adept_status _s = (expr);                 \
    if (_s != ADEPT_OK) return _s;            \
  } while (0)

// Brackets the kernel launched in its scope with timing events when timing is
// enabled (adept_timing_enable); a no-op otherwise.  `name` must be a literal.
class TimedLaunch {
 public:
  TimedLaunch(const char* name, hipStream_t s);
  ~TimedLaunch();
  TimedLaunch(const TimedLaunch&) = delete;
  TimedLaunch& operator=(const TimedLaunch&) = delete;

 private:
  const char* name_;
  hipStream_t s_;
  void* a_ = nullptr;
  void* b_ = nullptr;
};

// hipLaunchKernelGGL under a TimedLaunch named after the kernel expression.
#define ADEPT_LAUNCH(kernel, grid, block, smem, stream, ...)                 \
  do {                                                                       \
    ::adept::TimedLaunch _adept_tl(#kernel, stream);                         \
    hipLaunchKernelGGL(kernel, grid, block, smem, stream, __VA_ARGS__);      \
  } while (0)

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline hipStream_t as_stream(void* s) { return (hipStream_t)s; }
inline int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }

// ---------------------------------------------------------------------------
// internal launchers shared between translation units
// ---------------------------------------------------------------------------

// RMSNorm of gathered rows into a compact buffer:
// out[k] = x[rows ? rows[k] : k] / sqrt(mean(x^2) + eps) * gain, k < *n (or n_host).
adept_status rmsnorm_rows(adept_dtype dt, int d, float eps, const void* x, const int32_t* rows,
                          const int32_t* n_dev, int max_n, const void* gain, void* out,
                          hipStream_t s);

// GEMM epilogue kinds.
enum EpiKind {
  EPI_STORE = 0,   // C[k][n] (dtype or float) compact
  EPI_QKV = 1,     // RoPE on Q and K columns (none when rope_cos is NULL); Q -> q_out[k],
                   // K/V -> cache slot of rows[k]
  EPI_RESID = 2,   // out[rows[k]][n] = resid[rows[k]][n] + acc
  EPI_SWIGLU = 3,  // B = (gate, up) interleaved per 64 columns; out[k][n] = silu(g) * u
  EPI_KV = 4,      // K/V-only variant of EPI_QKV (KV generation, per-layer groups)
  EPI_GELU = 5,    // C[k][n] = gelu(acc) (exact erf form), dtype
  EPI_GELU_TANH = 6,  // C[k][n] = gelu(acc) (tanh approximation), dtype
};

struct GemmArgs {
  int M_max;              // grid bound on rows
  const int32_t* M_dev;   // device row count (nullable: M_max exact)
  int N, K;
  const void* A;          // [.][K] rows; row index = a_rows ? a_rows[m] : m
  const int32_t* a_rows;
  int64_t lda;
  const void* B;          // [N][K] (nn.Linear order)
  const void* B2;         // second matrix for SWIGLU (up); B is gate
  int64_t ldb;
  int epi;
  // epilogue operands
  void* C; int64_t ldc; int c_f32;
  const float* row_scale; // per-row scale of the accumulators (1/rms of the row), nullable
  const void* bias;       // [N] (dtype) added after the row scale, before the epilogue; nullable
  const int32_t* rows;    // token row of compact index k (QKV/RESID/KV)
  const void* resid;      // RESID source (may equal C)
  const int32_t* pos;     // [n_tok]
  const int32_t* slot;    // [n_tok] cache slot of a row (nullable: the row itself)
  const float* rope_cos; const float* rope_sin;
  int head_dim, d_q;
  void* q_out; void* k_cache; void* v_cache;   // caches already offset to the layer
  const char* name;       // timing label (string literal), nullable
  // f32 workspace of the skinny path (M_max <= 64: decode), nullable; used
  // when at least skinny_ws_bytes(N or 2N for SWIGLU, K) bytes
  float* skinny_ws; size_t skinny_ws_bytes;
  // grouped KV generation: per-layer bias stride, and A already in the
  // sorted row order (pre-normalised rows) instead of gathered by token row
  int64_t bias_layer_stride; int a_sorted;
  // per-row second A buffer (bf16 paths): token row r = a_rows[m] reads A2
  // instead of A when a_sel[r] & 1; nullable
  const void* A2; const int32_t* a_sel;
  // RESID on the skinny path only (gemm_skinny_row_norm says when), at most
  // one of: rinv_out[m] = 1/sqrt(mean(v^2) + row_eps), or ln_out[m] (bf16,
  // [M][N]) = (v - mean) / sqrt(var + row_eps), of each result row v (its
  // bf16 values); nullable.  Or exit (nullable): the GLOBAL exit test of
  // each result row (as adept_exit_test: flags, similarities, inertia update).
  float* rinv_out; void* ln_out; float row_eps;
  const struct RowExit* exit;
};
// The GLOBAL-metric exit test (Eq. 7-8) run by a residual epilogue over its
// result rows m (token rows rows[m]): flags and similarities by m, the
// inertia by token row.
struct RowExit {
  double delta;
  int layer, min_exit_layer, n_layers;
  float* inertia;               // [n_tok][N] f32, updated in place
  const int32_t* force_layer;   // nullable
  uint8_t* exit_flag;           // [M]
  double* sim_out;              // [M], nullable
};
size_t skinny_ws_bytes(int n_cols, int K);
// whether gemm() runs g on the skinny path and can fill g.rinv_out / g.ln_out
// or run g.exit
bool gemm_skinny_row_norm(const GemmArgs& g);

adept_status gemm(adept_dtype dt, const GemmArgs& g, hipStream_t s);       // bf16 MFMA path
// attention (csrc/attention.hip): adept_attend with a switch that can forbid
// the query-tile kernel (one query per sequence: decode)
size_t attend_workspace_bytes(int max_active, int n_seq, int n_heads, int head_dim, int s_max);
adept_status attend_dispatch(adept_dtype dt, int n_heads, int head_dim, float scale, int causal,
                             const void* q, const int32_t* rows, const int32_t* n_active,
                             int max_active, const int32_t* pos, const int32_t* seq, int n_seq,
                             const void* k_layer, const void* v_layer, int s_max,
                             const int32_t* key_len, const uint8_t* key_live, void* out,
                             void* workspace, size_t workspace_bytes, bool allow_tiles,
                             hipStream_t s);
adept_status gemm_f32(const GemmArgs& g, float* tmp, hipStream_t s);      // f32 + epilogue
adept_status gemm_f32_direct(const GemmArgs& g, hipStream_t s);           // f32, C = A B^T
adept_status gemm_kv_grouped(const GemmArgs& g, const int32_t* work, const int32_t* n_work,
                             int max_work, const int32_t* grp_m,
                             const int32_t* srows, int64_t b_layer_stride,
                             int64_t cache_layer_stride, hipStream_t s);
// out[k] = 1/sqrt(mean(x[rows[k]]^2) + eps) for k < min(*n_dev, max_n) (rows nullable: k).
adept_status row_rinv(adept_dtype dt, int d, float eps, const void* x, const int32_t* rows,
                      const int32_t* n_dev, int max_n, float* out, hipStream_t s);
// row_rinv of x1[row] where sel && (sel[row] & 1), else of x0[row]
adept_status row_rinv_sel(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                          const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                          int max_n, float* out, hipStream_t s);
adept_status rmsnorm_rows_sel(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                              const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                              int max_n, const void* gain, void* out, hipStream_t s);
// LayerNorm of gathered rows into a compact buffer (csrc/layernorm.hip):
// out[k] = (x - mean) / sqrt(var + eps) [* gain + bias] (gain NULL: no affine
// part), x = x1[row] when sel && (sel[row] & 1), else x0[row]; row = rows ? rows[k] : k.
adept_status layernorm_rows_sel(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                                const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                                int max_n, const void* gain, const void* bias, void* out,
                                hipStream_t s);
// the same, writing out[row] instead of out[k] when out_by_row (bf16 rows of
// a multiple of 8 elements up to 4096, 16-byte aligned; may run in place)
adept_status layernorm_rows_any(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                                const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                                int max_n, const void* gain, const void* bias, void* out,
                                bool out_by_row, hipStream_t s);

}  // namespace adept
