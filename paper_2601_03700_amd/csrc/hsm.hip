// Hidden State Mapper (Section 4.2; Appendix B, Table S1, Fig. S1) for the
// rows of exiting tokens, bf16.
//
// Per row k (token row rows[k]):
//   x_r = RMSNorm(z_r) * g0 for z = (s_i, s_{i-1}, inertia before layer i's
//         update), r = 0, 1, 2;
//   u   = conv_b + sum_r sum_t K[r][t] x_r[d + t - 1]   (3x3, padding (0, 1))
//   a   = W1 u + b1;  b = gelu(W2 gelu(a) + b2);  c = W3 b + b3
//   dd  = RMSNorm(c) * g1 + a;  e = W4 dd + b4;  s~ = RMSNorm(e) * g2 + u
// (GELU in its exact erf form.)  The input kernel (one wavefront per row,
// 16-byte loads) forms u; the four fully connected layers are MFMA GEMMs of the library
// over the compact rows (bias and GELU in their epilogues); a second
// row kernel applies GELU to a, and a norm-add row kernel forms dd and s~,
// the latter written to out[rows[k]] (out may be the current-state buffer:
// every read of it precedes that write in stream order).
#include "common.h"

namespace adept {
namespace {

constexpr int kRowWaves = 4;

struct Conv {
  float k[3][3];
  float b;
};

__device__ __forceinline__ float gelu_exact(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

// 8 consecutive bf16 as floats (one 16-byte load)
__device__ __forceinline__ void load8(const bf16* p, float* f) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f[2 * j] = __uint_as_float(q[j] << 16);
    f[2 * j + 1] = __uint_as_float(q[j] & 0xffff0000u);
  }
}

__device__ __forceinline__ void store8(bf16* p, const float* f) {
  *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]),
                                            pack_bf16x2(f[4], f[5]), pack_bf16x2(f[6], f[7]));
}

// u[k] from the three states of row rows[k].  post != 0: the inertia buffer
// already holds layer i's update (inertia += s_i/|s_i|), which is taken back.
// Each lane takes 8 consecutive elements per step (16-byte loads); the
// convolution's neighbours one element outside a lane's 8 are read directly.
__global__ __launch_bounds__(64 * kRowWaves) void hsm_input_kernel(
    int d, float eps, const int32_t* __restrict__ rows, const int32_t* __restrict__ n_rows,
    int max_rows, const bf16* __restrict__ h_cur, const bf16* __restrict__ h_prev,
    const float* __restrict__ inertia, int post, const bf16* __restrict__ g0, Conv cv,
    bf16* __restrict__ u) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (k >= min(*n_rows, max_rows)) return;
  const int64_t row = rows[k];
  const bf16* z0 = h_cur + row * d;
  const bf16* z1 = h_prev + row * d;
  const float* zi = inertia + row * d;
  double s0 = 0.0, s1 = 0.0;
  for (int e = lane * 8; e < d; e += 512) {
    float a[8], b[8];
    load8(z0 + e, a);
    load8(z1 + e, b);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      s0 += (double)a[j] * a[j];
      s1 += (double)b[j] * b[j];
    }
  }
  s0 = wave_sum_f64(s0);
  s1 = wave_sum_f64(s1);
  const float inv0 = (post && s0 > 0.0) ? (float)(1.0 / sqrt(s0)) : 0.0f;
  // 8 inertia values from element e, with the update taken back
  auto load_i8 = [&](int e, float* c) {
    const float4 v0 = *reinterpret_cast<const float4*>(zi + e);
    const float4 v1 = *reinterpret_cast<const float4*>(zi + e + 4);
    float a[8];
    load8(z0 + e, a);
    const float iv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) c[j] = iv[j] - a[j] * inv0;
  };
  double s2 = 0.0;
  for (int e = lane * 8; e < d; e += 512) {
    float c[8];
    load_i8(e, c);
#pragma unroll
    for (int j = 0; j < 8; ++j) s2 += (double)c[j] * c[j];
  }
  s2 = wave_sum_f64(s2);
  const float r[3] = {(float)(1.0 / sqrt(s0 / d + eps)), (float)(1.0 / sqrt(s1 / d + eps)),
                      (float)(1.0 / sqrt(s2 / d + eps))};
  // one normalised element outside the lane's 8 (zero past either end)
  auto x1 = [&](int rr, int e) -> float {
    if (e < 0 || e >= d) return 0.0f;
    const float v = rr == 0 ? bf2f(z0[e]) : (rr == 1 ? bf2f(z1[e]) : zi[e] - bf2f(z0[e]) * inv0);
    return v * r[rr] * bf2f(g0[e]);
  };
  bf16* uo = u + (int64_t)k * d;
  for (int e = lane * 8; e < d; e += 512) {
    float x[3][10];   // elements e-1 .. e+8 of the three normalised rows
    float gv[8], a[8];
    load8(g0 + e, gv);
    load8(z0 + e, a);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[0][j + 1] = a[j] * r[0] * gv[j];
    load8(z1 + e, a);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[1][j + 1] = a[j] * r[1] * gv[j];
    load_i8(e, a);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[2][j + 1] = a[j] * r[2] * gv[j];
#pragma unroll
    for (int rr = 0; rr < 3; ++rr) {
      x[rr][0] = x1(rr, e - 1);
      x[rr][9] = x1(rr, e + 8);
    }
    float o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float acc = cv.b;
#pragma unroll
      for (int rr = 0; rr < 3; ++rr)
#pragma unroll
        for (int t = 0; t < 3; ++t) acc = fmaf(cv.k[rr][t], x[rr][j + t], acc);
      o[j] = acc;
    }
    store8(uo + e, o);
  }
}

// y[k] = gelu(x[k]) over [rows][w] (compact rows, device count).
__global__ __launch_bounds__(256) void hsm_gelu_kernel(int w, const int32_t* __restrict__ n_rows,
                                                       int max_rows, const bf16* __restrict__ x,
                                                       bf16* __restrict__ y) {
  const int64_t n = (int64_t)min(*n_rows, max_rows) * w;
  for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8; i < n;
       i += (int64_t)gridDim.x * 256 * 8) {
    // w is a multiple of 8: one 16-byte vector per thread and step
    float f[8];
    load8(x + i, f);
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = gelu_exact(f[j]);
    store8(y + i, f);
  }
}

// out[dst(k)] = x[k] / rms(x[k]) * g + skip[k] over width w (one wavefront
// per row, 8 elements per lane and step); dst(k) = rows[k] when rows is
// given, else k.
__global__ __launch_bounds__(64 * kRowWaves) void hsm_norm_add_kernel(
    int w, float eps, const int32_t* __restrict__ rows, const int32_t* __restrict__ n_rows,
    int max_rows, const bf16* __restrict__ x, const bf16* __restrict__ g,
    const bf16* __restrict__ skip, bf16* out) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (k >= min(*n_rows, max_rows)) return;
  const bf16* xr = x + (int64_t)k * w;
  double ss = 0.0;
  for (int e = lane * 8; e < w; e += 512) {
    float f[8];
    load8(xr + e, f);
#pragma unroll
    for (int j = 0; j < 8; ++j) ss += (double)f[j] * f[j];
  }
  ss = wave_sum_f64(ss);
  const float rinv = (float)(1.0 / sqrt(ss / w + eps));
  const bf16* sr = skip + (int64_t)k * w;
  bf16* o = out + (int64_t)(rows ? rows[k] : k) * w;
  for (int e = lane * 8; e < w; e += 512) {
    float f[8], gv[8], sv[8];
    load8(xr + e, f);
    load8(g + e, gv);
    load8(sr + e, sv);
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = f[j] * rinv * gv[j] + sv[j];
    store8(o + e, f);
  }
}

struct HsmWs {
  bf16 *u, *a, *ga, *gb, *c, *e;
  size_t total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

HsmWs carve(int d, int max_rows, void* base) {
  HsmWs w{};
  char* p = (char*)base;
  size_t off = 0;
  const size_t m = (size_t)max_rows;
  auto take = [&](size_t cols) {
    bf16* q = (bf16*)(p + off);
    off += align256(m * cols * sizeof(bf16));
    return q;
  };
  w.u = take(d);
  w.a = take(4 * (size_t)d);
  w.ga = take(4 * (size_t)d);   // gelu(a), later the first Norm+Add
  w.gb = take(8 * (size_t)d);
  w.c = take(4 * (size_t)d);
  w.e = take(d);
  w.total = off;
  return w;
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_hsm_workspace_bytes(int d_model, int max_rows) {
  if (d_model <= 0 || max_rows <= 0) return 0;
  return carve(d_model, max_rows, nullptr).total;
}

extern "C" adept_status adept_hsm_forward(adept_dtype dt, int d_model, float eps,
                                          const adept_hsm_weights* w, const int32_t* rows,
                                          const int32_t* n_rows, int max_rows,
                                          const void* h_cur, const void* h_prev,
                                          const float* inertia, int inertia_updated, void* out,
                                          void* workspace, size_t workspace_bytes,
                                          void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_BF16, "hsm_forward: bf16 only");
  ADEPT_REQUIRE(w != nullptr, "hsm_forward: weights are NULL");
  ADEPT_REQUIRE(d_model > 0 && d_model % 256 == 0, "hsm_forward: d_model %d not a multiple of 256",
                d_model);
  ADEPT_REQUIRE(max_rows >= 0, "hsm_forward: max_rows < 0");
  ADEPT_REQUIRE(rows && n_rows && h_cur && h_prev && inertia && out, "hsm_forward: NULL tensor");
  ADEPT_REQUIRE(w->g0 && w->w1 && w->b1 && w->w2 && w->b2 && w->w3 && w->b3 && w->g1 &&
                    w->w4 && w->b4 && w->g2,
                "hsm_forward: NULL weight");
  ADEPT_REQUIRE(aligned16(w->w1) && aligned16(w->w2) && aligned16(w->w3) && aligned16(w->w4) &&
                    aligned16(w->g0) && aligned16(w->g1) && aligned16(w->g2) &&
                    aligned16(h_cur) && aligned16(h_prev) && aligned16(inertia) &&
                    aligned16(out) && aligned16(workspace),
                "hsm_forward: weights, states and workspace must be 16-byte aligned");
  if (max_rows == 0) return ADEPT_OK;
  const size_t need = adept_hsm_workspace_bytes(d_model, max_rows);
  if (!workspace || workspace_bytes < need) {
    set_error("hsm_forward: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  hipStream_t s = as_stream(stream);
  const int D = d_model;
  HsmWs ws = carve(D, max_rows, workspace);
  Conv cv;
  for (int r = 0; r < 3; ++r)
    for (int t = 0; t < 3; ++t) cv.k[r][t] = w->conv[r][t];
  cv.b = w->conv_bias;
  const dim3 row_grid(ceil_div(max_rows, kRowWaves)), row_block(64 * kRowWaves);
  ADEPT_LAUNCH(hsm_input_kernel, row_grid, row_block, 0, s, D, eps, rows, n_rows, max_rows,
               (const bf16*)h_cur, (const bf16*)h_prev, inertia, inertia_updated,
               (const bf16*)w->g0, cv, ws.u);
  ADEPT_CHECK_LAUNCH("hsm_input");
  auto fc = [&](const void* A, int K, const void* B, const void* bias, int N, int epi, void* C,
                const char* name) {
    GemmArgs g{};
    g.M_max = max_rows; g.M_dev = n_rows; g.N = N; g.K = K;
    g.A = A; g.lda = K; g.B = B; g.ldb = K; g.epi = epi;
    g.C = C; g.ldc = N; g.bias = bias; g.name = name;
    return gemm(ADEPT_BF16, g, s);
  };
  ADEPT_TRY(fc(ws.u, D, w->w1, w->b1, 4 * D, EPI_STORE, ws.a, "hsm_fc1"));
  ADEPT_LAUNCH(hsm_gelu_kernel, dim3(std::min(ceil_div((int64_t)max_rows * 4 * D, 256 * 8), 4096)),
               dim3(256), 0, s, 4 * D, n_rows, max_rows, ws.a, ws.ga);
  ADEPT_CHECK_LAUNCH("hsm_gelu");
  ADEPT_TRY(fc(ws.ga, 4 * D, w->w2, w->b2, 8 * D, EPI_GELU, ws.gb, "hsm_fc2"));
  ADEPT_TRY(fc(ws.gb, 8 * D, w->w3, w->b3, 4 * D, EPI_STORE, ws.c, "hsm_fc3"));
  ADEPT_LAUNCH(hsm_norm_add_kernel, row_grid, row_block, 0, s, 4 * D, eps, nullptr, n_rows,
               max_rows, ws.c, (const bf16*)w->g1, ws.a, ws.ga);
  ADEPT_CHECK_LAUNCH("hsm_norm_add_mid");
  ADEPT_TRY(fc(ws.ga, 4 * D, w->w4, w->b4, D, EPI_STORE, ws.e, "hsm_fc4"));
  ADEPT_LAUNCH(hsm_norm_add_kernel, row_grid, row_block, 0, s, D, eps, rows, n_rows, max_rows,
               ws.e, (const bf16*)w->g2, ws.u, (bf16*)out);
  return launch_status("hsm_norm_add_out");
}
