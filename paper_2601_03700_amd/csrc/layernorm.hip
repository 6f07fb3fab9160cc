// Support steps of the LayerNorm decoder family (GPT-2 style: LayerNorm with
// bias, learned absolute positions, biased projections, head tied to the
// token embedding; the GPT2-XL shape of Section 5):
//
//  * LayerNorm of gathered rows, f32 statistics, optionally affine.  The
//    layer step normalises without the affine part: the gain gamma is folded
//    into the columns of the projection that follows and the shift beta
//    into its bias, (xh gamma + beta) W^T + b = xh (W diag gamma)^T + (b + W beta),
//    so one folded copy of Wk / Wv serves both the layer's own K / V and the
//    decoupled KV generation of exited tokens (Eq. 9), as the RMSNorm gains
//    of the other family do.
//  * the embedding with learned positions, the bias fold, the final
//    LayerNorm and the tied LM head.
#include <algorithm>

#include "common.h"

namespace adept {
namespace {

// One wave per row k < min(*n_dev, max_n): x = (sel && (sel[row] & 1)) ?
// x1[row] : x0[row], row = rows ? rows[k] : k;
// out[k] = (x - mean) / sqrt(var + eps) [* gain + bias].  Mean and variance
// in f32 over two passes (the second re-reads the row from cache).
template <typename T>
__global__ __launch_bounds__(256) void layernorm_rows_kernel(
    int d, float eps, const T* __restrict__ x0, const T* __restrict__ x1,
    const int32_t* __restrict__ sel, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_dev, int max_n, const T* __restrict__ gain,
    const T* __restrict__ bias, T* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(*n_dev, max_n) : max_n;
  if (k >= n) return;
  const int row = rows ? rows[k] : k;
  const T* x = ((sel && (sel[row] & 1)) ? x1 : x0) + (int64_t)row * d;
  float s = 0.0f;
  for (int c = lane; c < d; c += 64) s += ld(x + c);
  const float mean = wave_sum_f32(s) / (float)d;
  float v = 0.0f;
  for (int c = lane; c < d; c += 64) {
    const float t = ld(x + c) - mean;
    v = fmaf(t, t, v);
  }
  const float r = 1.0f / sqrtf(wave_sum_f32(v) / (float)d + eps);
  T* o = out + (int64_t)k * d;
  for (int c = lane; c < d; c += 64) {
    float y = (ld(x + c) - mean) * r;
    if (gain) y = fmaf(y, ld(gain + c), bias ? ld(bias + c) : 0.0f);
    st(o + c, y);
  }
}

// The same for bf16 rows held in registers (layernorm_row_vec, shared with
// the layer step); out row = out_by_row ? row : k (in place when
// out == x0 == x1).
template <int R>
__global__ __launch_bounds__(256) void layernorm_vec_kernel(
    int d, float eps, const bf16* x0, const bf16* x1, const int32_t* __restrict__ sel,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ n_dev, int max_n,
    const bf16* __restrict__ gain, const bf16* __restrict__ bias, bf16* out, int out_by_row) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(*n_dev, max_n) : max_n;
  if (k >= n) return;
  const int row = rows ? rows[k] : k;
  const bf16* x = ((sel && (sel[row] & 1)) ? x1 : x0) + (int64_t)row * d;
  layernorm_row_vec<R>(x, d, eps, gain, bias, out + (int64_t)(out_by_row ? row : k) * d, lane);
}

// h0[k][c] = wte[ids[k]][c] + wpe[pos[k]][c] (ids and positions clamped
// into the tables), summed in f32 and rounded once.
template <typename T>
__global__ void embed_positions_kernel(int n, int d, int vocab, int max_pos,
                                       const int32_t* __restrict__ ids,
                                       const int32_t* __restrict__ pos,
                                       const T* __restrict__ wte, const T* __restrict__ wpe,
                                       T* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * d) return;
  const int k = (int)(idx / d), c = (int)(idx % d);
  const int64_t id = min(max(ids[k], 0), vocab - 1);
  const int64_t p = min(max(pos[k], 0), max_pos - 1);
  st(out + idx, ld(wte + id * d + c) + ld(wpe + p * d + c));
}

// bias[l][o] += sum_c w[l][o][c] * shift[l][c]: one wave per (l, o), the
// dot product in f32, rounded once into the bias.
template <typename T>
__global__ __launch_bounds__(256) void fold_bias_kernel(int rows, int cols,
                                                        const T* __restrict__ w,
                                                        int64_t mat_stride,
                                                        const T* __restrict__ shift,
                                                        int64_t shift_stride, T* __restrict__ bias,
                                                        int64_t bias_stride) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = blockIdx.y;
  if (o >= rows) return;
  const T* wr = w + (int64_t)l * mat_stride + (int64_t)o * cols;
  const T* sh = shift + (int64_t)l * shift_stride;
  float a = 0.0f;
  for (int c = lane; c < cols; c += 64) a = fmaf(ld(wr + c), ld(sh + c), a);
  a = wave_sum_f32(a);
  if (lane == 0) {
    T* b = bias + (int64_t)l * bias_stride + o;
    st(b, ld(b) + a);
  }
}

}  // namespace

adept_status layernorm_rows_any(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                                const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                                int max_n, const void* gain, const void* bias, void* out,
                                bool out_by_row, hipStream_t s) {
  if (max_n <= 0) return ADEPT_OK;
  dim3 grid(ceil_div(max_n, 4)), block(256);
  const bool vec = dt == ADEPT_BF16 && d % 8 == 0 && d <= 64 * 8 * 8 && aligned16(x0) &&
                   aligned16(x1) && aligned16(out) && (!gain || (aligned16(gain) && bias &&
                                                                 aligned16(bias)));
  if (vec) {
    const int chunks = ceil_div(d / 8, 64);
    const bf16 *a0 = (const bf16*)x0, *a1 = (const bf16*)x1;
    const bf16 *g = (const bf16*)gain, *b = (const bf16*)bias;
    const int obr = out_by_row ? 1 : 0;
    if (chunks <= 1)
      ADEPT_LAUNCH(layernorm_vec_kernel<1>, grid, block, 0, s, d, eps, a0, a1, sel, rows, n_dev,
                   max_n, g, b, (bf16*)out, obr);
    else if (chunks <= 2)
      ADEPT_LAUNCH(layernorm_vec_kernel<2>, grid, block, 0, s, d, eps, a0, a1, sel, rows, n_dev,
                   max_n, g, b, (bf16*)out, obr);
    else if (chunks <= 4)
      ADEPT_LAUNCH(layernorm_vec_kernel<4>, grid, block, 0, s, d, eps, a0, a1, sel, rows, n_dev,
                   max_n, g, b, (bf16*)out, obr);
    else
      ADEPT_LAUNCH(layernorm_vec_kernel<8>, grid, block, 0, s, d, eps, a0, a1, sel, rows, n_dev,
                   max_n, g, b, (bf16*)out, obr);
    return launch_status("layernorm_rows");
  }
  if (out_by_row) {
    set_error("layernorm: the in-place form needs bf16 rows of a multiple of 8 up to 4096, "
              "16-byte aligned");
    return ADEPT_E_UNSUPPORTED;
  }
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(layernorm_rows_kernel<bf16>, grid, block, 0, s, d, eps, (const bf16*)x0,
                 (const bf16*)x1, sel, rows, n_dev, max_n, (const bf16*)gain, (const bf16*)bias,
                 (bf16*)out);
  else
    ADEPT_LAUNCH(layernorm_rows_kernel<float>, grid, block, 0, s, d, eps, (const float*)x0,
                 (const float*)x1, sel, rows, n_dev, max_n, (const float*)gain,
                 (const float*)bias, (float*)out);
  return launch_status("layernorm_rows");
}

adept_status layernorm_rows_sel(adept_dtype dt, int d, float eps, const void* x0, const void* x1,
                                const int32_t* sel, const int32_t* rows, const int32_t* n_dev,
                                int max_n, const void* gain, const void* bias, void* out,
                                hipStream_t s) {
  return layernorm_rows_any(dt, d, eps, x0, x1, sel, rows, n_dev, max_n, gain, bias, out, false,
                            s);
}

}  // namespace adept

using namespace adept;

extern "C" adept_status adept_embed_positions(adept_dtype dt, int n, int d_model, int vocab,
                                              int max_pos, const int32_t* ids,
                                              const int32_t* pos, const void* wte,
                                              const void* wpe, void* h0, void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "embed_positions: bad dtype");
  ADEPT_REQUIRE(n >= 0 && d_model > 0 && vocab > 0 && max_pos > 0, "embed_positions: bad sizes");
  ADEPT_REQUIRE(ids && pos && wte && wpe && h0, "embed_positions: NULL tensor");
  if (n == 0) return ADEPT_OK;
  const int64_t total = (int64_t)n * d_model;
  dim3 grid((unsigned)((total + 255) / 256));
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(embed_positions_kernel<bf16>, grid, dim3(256), 0, as_stream(stream), n,
                 d_model, vocab, max_pos, ids, pos, (const bf16*)wte, (const bf16*)wpe,
                 (bf16*)h0);
  else
    ADEPT_LAUNCH(embed_positions_kernel<float>, grid, dim3(256), 0, as_stream(stream), n,
                 d_model, vocab, max_pos, ids, pos, (const float*)wte, (const float*)wpe,
                 (float*)h0);
  return launch_status("embed_positions");
}

extern "C" adept_status adept_fold_bias(adept_dtype dt, int n_mats, int rows, int cols,
                                        const void* w, int64_t mat_stride, const void* shift,
                                        int64_t shift_stride, void* bias, int64_t bias_stride,
                                        void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "fold_bias: bad dtype");
  ADEPT_REQUIRE(n_mats >= 0 && n_mats <= 65535 && rows >= 0 && cols > 0, "fold_bias: bad sizes");
  ADEPT_REQUIRE(mat_stride >= (int64_t)rows * cols && shift_stride >= 0 && bias_stride >= rows,
                "fold_bias: strides smaller than a matrix / bias row");
  ADEPT_REQUIRE(w && shift && bias, "fold_bias: NULL tensor");
  if (n_mats == 0 || rows == 0) return ADEPT_OK;
  dim3 grid(ceil_div(rows, 4), n_mats);
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(fold_bias_kernel<bf16>, grid, dim3(256), 0, as_stream(stream), rows, cols,
                 (const bf16*)w, mat_stride, (const bf16*)shift, shift_stride, (bf16*)bias,
                 bias_stride);
  else
    ADEPT_LAUNCH(fold_bias_kernel<float>, grid, dim3(256), 0, as_stream(stream), rows, cols,
                 (const float*)w, mat_stride, (const float*)shift, shift_stride, (float*)bias,
                 bias_stride);
  return launch_status("fold_bias");
}

extern "C" adept_status adept_final_logits_layernorm(adept_dtype dt, int d_model, int vocab,
                                                     float eps, const void* h0_buf,
                                                     const void* h1_buf,
                                                     const int32_t* exit_layer,
                                                     const int32_t* rows, const int32_t* n_rows,
                                                     int max_rows, const void* ln_g,
                                                     const void* ln_b, const void* lm_head,
                                                     void* x_norm, float* logits, void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_BF16, "final_logits_layernorm: bf16 only");
  ADEPT_REQUIRE(d_model > 0 && d_model % 64 == 0 && vocab > 0 && vocab % 64 == 0 &&
                    max_rows >= 0,
                "final_logits_layernorm: d_model and vocab must be multiples of 64");
  ADEPT_REQUIRE(h0_buf && h1_buf && exit_layer && rows && ln_g && ln_b && lm_head && x_norm &&
                    logits,
                "final_logits_layernorm: NULL tensor");
  if (max_rows == 0) return ADEPT_OK;
  hipStream_t s = as_stream(stream);
  ADEPT_TRY(layernorm_rows_sel(dt, d_model, eps, h0_buf, h1_buf, exit_layer, rows, n_rows,
                               max_rows, ln_g, ln_b, x_norm, s));
  GemmArgs g{};
  g.M_max = max_rows; g.M_dev = n_rows; g.N = vocab; g.K = d_model;
  g.A = x_norm; g.lda = d_model; g.B = lm_head; g.ldb = d_model;
  g.epi = EPI_STORE; g.C = logits; g.ldc = vocab; g.c_f32 = 1; g.name = "gemm_lm_head";
  return gemm(dt, g, s);
}
