// Support operations around the hot path: error reporting, the rotary table,
// row-gathered RMSNorm, embedding gather, final norm + LM head, greedy argmax.
#include <algorithm>
#include <cstdarg>

#include "common.h"

namespace adept {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

adept_status launch_status(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("%s: %s", what, hipGetErrorString(e));
    return ADEPT_E_HIP;
  }
  return ADEPT_OK;
}

namespace {

__global__ void rope_table_kernel(int max_pos, int half, double theta, float* cs, float* sn) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)max_pos * half) return;
  const int p = (int)(idx / half), k = (int)(idx % half);
  const double inv_freq = pow(theta, -2.0 * (double)k / (double)(2 * half));
  const double ang = (double)p * inv_freq;
  cs[idx] = (float)cos(ang);
  sn[idx] = (float)sin(ang);
}

// One wave per row: out[k] = x[row] * rsqrt(mean(x^2) + eps) * gain, row =
// rows ? rows[k] : k, with x taken from x1 when sel && (sel[row] & 1).
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(int d, float eps, const T* __restrict__ x0,
                                                      const T* __restrict__ x1,
                                                      const int32_t* __restrict__ sel,
                                                      const int32_t* __restrict__ rows,
                                                      const int32_t* __restrict__ n_dev, int max_n,
                                                      const T* __restrict__ gain,
                                                      T* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(*n_dev, max_n) : max_n;
  if (k >= n) return;
  const int row = rows ? rows[k] : k;
  const T* x = (sel && (sel[row] & 1)) ? x1 : x0;
  x += (int64_t)row * d;
  float ss = 0.0f;
  for (int c = lane; c < d; c += 64) {
    const float v = ld(x + c);
    ss = fmaf(v, v, ss);
  }
  ss = wave_sum_f32(ss);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  T* o = out + (int64_t)k * d;
  for (int c = lane; c < d; c += 64) st(o + c, ld(x + c) * r * ld(gain + c));
}

// One wave per row: out[k] = 1/sqrt(mean(x[row]^2) + eps), x = x1 when
// sel && (sel[row] & 1), else x0.
template <typename T>
__global__ __launch_bounds__(256) void row_rinv_kernel(int d, float eps, const T* __restrict__ x0,
                                                       const T* __restrict__ x1,
                                                       const int32_t* __restrict__ sel,
                                                       const int32_t* __restrict__ rows,
                                                       const int32_t* __restrict__ n_dev,
                                                       int max_n, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(*n_dev, max_n) : max_n;
  if (k >= n) return;
  const int row = rows ? rows[k] : k;
  const T* xr = ((sel && (sel[row] & 1)) ? x1 : x0) + (int64_t)row * d;
  const float r = row_rinv_wave(xr, d, eps, lane);
  if (lane == 0) out[k] = r;
}

// w[l][o][c] *= gain[l][c] (in place, rounded to the element type).
template <typename T>
__global__ void fold_gain_kernel(int rows, int cols, T* __restrict__ w, int64_t mat_stride,
                                 const T* __restrict__ gain, int64_t gain_stride) {
  const int l = blockIdx.y;
  T* wm = w + (int64_t)l * mat_stride;
  const T* g = gain + (int64_t)l * gain_stride;
  const int64_t total = (int64_t)rows * cols;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x)
    st(wm + e, ld(wm + e) * ld(g + e % cols));
}

template <typename T>
__global__ void embed_kernel(int n, int d, int vocab, const int32_t* __restrict__ ids,
                             const T* __restrict__ table, T* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * d) return;
  const int k = (int)(idx / d), c = (int)(idx % d);
  int id = ids[k];
  id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
  out[idx] = table[(int64_t)id * d + c];
}

__global__ __launch_bounds__(256) void argmax_kernel(int vocab, const float* __restrict__ logits,
                                                     int32_t* __restrict__ out) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const float* r = logits + (int64_t)blockIdx.x * vocab;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int v = threadIdx.x; v < vocab; v += 256) {
    const float x = r[v];
    if (x > bv || (x == bv && v < bi)) { bv = x; bi = v; }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
  }
  if ((threadIdx.x & 63) == 0) { sv[threadIdx.x >> 6] = bv; si[threadIdx.x >> 6] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (sv[w] > bv || (sv[w] == bv && si[w] < bi)) { bv = sv[w]; bi = si[w]; }
    out[blockIdx.x] = bi;
  }
}

}  // namespace

adept_status rmsnorm_rows_sel(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                              const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                              int max_n, const void* gain, void* out, hipStream_t s) {
  if (max_n <= 0) return ADEPT_OK;
  dim3 grid(ceil_div(max_n, 4)), block(256);
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(rmsnorm_kernel<bf16>, grid, block, 0, s, d, eps, (const bf16*)x0,
                       (const bf16*)x1, sel, rows, n_dev, max_n, (const bf16*)gain, (bf16*)out);
  else
    ADEPT_LAUNCH(rmsnorm_kernel<float>, grid, block, 0, s, d, eps, (const float*)x0,
                       (const float*)x1, sel, rows, n_dev, max_n, (const float*)gain,
                       (float*)out);
  return launch_status("rmsnorm");
}

adept_status rmsnorm_rows(adept_dtype dt, int d, float eps, const void* x, const int32_t* rows,
                          const int32_t* n_dev, int max_n, const void* gain, void* out,
                          hipStream_t s) {
  return rmsnorm_rows_sel(dt, d, eps, x, x, nullptr, rows, n_dev, max_n, gain, out, s);
}

adept_status row_rinv_sel(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                          const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                          int max_n, float* out, hipStream_t s) {
  if (max_n <= 0) return ADEPT_OK;
  dim3 grid(ceil_div(max_n, 4)), block(256);
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(row_rinv_kernel<bf16>, grid, block, 0, s, d, eps, (const bf16*)x0,
                 (const bf16*)x1, sel, rows, n_dev, max_n, out);
  else
    ADEPT_LAUNCH(row_rinv_kernel<float>, grid, block, 0, s, d, eps, (const float*)x0,
                 (const float*)x1, sel, rows, n_dev, max_n, out);
  return launch_status("row_rinv");
}

adept_status row_rinv(adept_dtype dt, int d, float eps, const void* x, const int32_t* rows,
                      const int32_t* n_dev, int max_n, float* out, hipStream_t s) {
  return row_rinv_sel(dt, d, eps, x, x, nullptr, rows, n_dev, max_n, out, s);
}

}  // namespace adept

using namespace adept;

extern "C" int adept_abi_version(void) { return ADEPT_ABI_VERSION; }

extern "C" const char* adept_last_error(void) { return g_last_error.c_str(); }

extern "C" adept_status adept_rope_table(int max_pos, int head_dim, double theta, float* cos_out,
                                         float* sin_out, void* stream) {
  ADEPT_REQUIRE(max_pos > 0 && head_dim > 0 && head_dim % 2 == 0, "rope_table: bad sizes");
  ADEPT_REQUIRE(theta > 0.0, "rope_table: theta must be positive");
  ADEPT_REQUIRE(cos_out && sin_out, "rope_table: NULL tensor");
  const int half = head_dim / 2;
  const int64_t total = (int64_t)max_pos * half;
  ADEPT_LAUNCH(rope_table_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                     as_stream(stream), max_pos, half, theta, cos_out, sin_out);
  return launch_status("rope_table");
}

extern "C" adept_status adept_fold_gain(adept_dtype dt, int n_mats, int rows, int cols, void* w,
                                        int64_t mat_stride, const void* gain,
                                        int64_t gain_stride, void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "fold_gain: bad dtype");
  ADEPT_REQUIRE(n_mats >= 0 && rows >= 0 && cols > 0 && n_mats <= 65535, "fold_gain: bad sizes");
  ADEPT_REQUIRE(mat_stride >= (int64_t)rows * cols && gain_stride >= cols,
                "fold_gain: strides smaller than a matrix / gain row");
  ADEPT_REQUIRE(w && gain, "fold_gain: NULL tensor");
  if (n_mats == 0 || rows == 0) return ADEPT_OK;
  const int64_t total = (int64_t)rows * cols;
  const int bx = (int)std::min<int64_t>((total + 255) / 256, 8192);
  dim3 grid(bx, n_mats);
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(fold_gain_kernel<bf16>, grid, dim3(256), 0, as_stream(stream), rows, cols,
                 (bf16*)w, mat_stride, (const bf16*)gain, gain_stride);
  else
    ADEPT_LAUNCH(fold_gain_kernel<float>, grid, dim3(256), 0, as_stream(stream), rows, cols,
                 (float*)w, mat_stride, (const float*)gain, gain_stride);
  return launch_status("fold_gain");
}

extern "C" adept_status adept_embed(adept_dtype dt, int n, int d_model, int vocab,
                                    const int32_t* ids, const void* embed, void* h0,
                                    void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "embed: bad dtype");
  ADEPT_REQUIRE(n >= 0 && d_model > 0 && vocab > 0, "embed: bad sizes");
  ADEPT_REQUIRE(ids && embed && h0, "embed: NULL tensor");
  if (n == 0) return ADEPT_OK;
  const int64_t total = (int64_t)n * d_model;
  dim3 grid((unsigned)((total + 255) / 256));
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(embed_kernel<bf16>, grid, dim3(256), 0, as_stream(stream), n, d_model,
                       vocab, ids, (const bf16*)embed, (bf16*)h0);
  else
    ADEPT_LAUNCH(embed_kernel<float>, grid, dim3(256), 0, as_stream(stream), n, d_model,
                       vocab, ids, (const float*)embed, (float*)h0);
  return launch_status("embed");
}

extern "C" adept_status adept_argmax(int n, int vocab, const float* logits, int32_t* out,
                                     void* stream) {
  ADEPT_REQUIRE(n >= 0 && vocab > 0 && logits && out, "argmax: bad arguments");
  if (n == 0) return ADEPT_OK;
  ADEPT_LAUNCH(argmax_kernel, dim3(n), dim3(256), 0, as_stream(stream), vocab, logits, out);
  return launch_status("argmax");
}

extern "C" adept_status adept_final_logits(adept_dtype dt, int d_model, int vocab, float eps,
                                           const void* h0_buf, const void* h1_buf,
                                           const int32_t* exit_layer, const int32_t* rows,
                                           const int32_t* n_rows, int max_rows,
                                           const void* final_norm, const void* lm_head,
                                           void* x_norm, float* logits, void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "final_logits: bad dtype");
  ADEPT_REQUIRE(d_model > 0 && vocab > 0 && max_rows >= 0, "final_logits: bad sizes");
  ADEPT_REQUIRE(h0_buf && h1_buf && exit_layer && rows && final_norm && lm_head && x_norm &&
                    logits,
                "final_logits: NULL tensor");
  if (max_rows == 0) return ADEPT_OK;
  hipStream_t s = as_stream(stream);
  ADEPT_TRY(rmsnorm_rows_sel(dt, d_model, eps, h0_buf, h1_buf, exit_layer, rows, n_rows, max_rows,
                             final_norm, x_norm, s));
  GemmArgs g{};
  g.M_max = max_rows; g.M_dev = n_rows; g.N = vocab; g.K = d_model;
  g.A = x_norm; g.lda = d_model; g.B = lm_head; g.ldb = d_model;
  g.epi = EPI_STORE; g.C = logits; g.ldc = vocab; g.c_f32 = 1; g.name = "gemm_lm_head";
  if (dt == ADEPT_BF16) return gemm(dt, g, s);
  // f32: plain GEMM straight into the logits (EPI_STORE needs no scratch)
  return gemm_f32_direct(g, s);
}

namespace adept {
namespace {
__global__ void token_init_kernel(int n_tok, int n_layers, int d, int32_t* active, int32_t* n_active,
                                  int32_t* exit_layer, float* inertia) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // grid-stride: the grid is capped, the row count is not
  for (int64_t j = idx; j < n_tok; j += stride) {
    active[j] = (int32_t)j;
    exit_layer[j] = n_layers;
  }
  if (idx == 0) *n_active = n_tok;
  if (inertia) {
    for (int64_t e = idx; e < (int64_t)n_tok * d; e += stride) inertia[e] = 0.0f;
  }
}
}  // namespace
}  // namespace adept

extern "C" adept_status adept_token_init(int n_tok, int n_layers, int d_model, int32_t* active,
                                         int32_t* n_active, int32_t* exit_layer, float* inertia,
                                         void* stream) {
  ADEPT_REQUIRE(n_tok >= 0 && n_layers >= 1 && d_model > 0, "token_init: bad sizes");
  ADEPT_REQUIRE(active && n_active && exit_layer, "token_init: NULL tensor");
  const int blocks = std::max(1, std::min(ceil_div(std::max(n_tok, 1), 256), 4096));
  ADEPT_LAUNCH(token_init_kernel, dim3(blocks), dim3(256), 0, as_stream(stream), n_tok,
                     n_layers, d_model, active, n_active, exit_layer, inertia);
  return launch_status("token_init");
}
