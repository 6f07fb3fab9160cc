// Decoupled KV generation (Section 4, Eq. 6; Section 4.3, Eq. 9).
//
// bf16: a one-workgroup plan sorts the listed rows by exit layer (counting
// sort over the N+1 layer bins), so that for every skipped layer r the rows
// with i* < r form a prefix of length grp_m[r]; it then lists the work items
// (r, 256-row tile).  A wave-per-row pass computes each sorted row's
// 1/sqrt(mean s^2 + eps).  The grouped MFMA GEMM (gemm.hip) does the rest in
// one launch.  The norm is split: layer r's gain multiplies the columns of
// W_r beforehand (adept_fold_gain: (s * g) W^T = s (W diag g)^T), and the
// row factor 1/rms(s) scales the accumulators; RoPE on K in the epilogue,
// K/V stored straight into cache[r][slot].
//
// f32 (small configurations): one workgroup per (row, layer) pair computes
// the normalised state in LDS and the 2*H*hd dot products directly.
//
// adept_kv_generate_noalloc runs the same kernels with their scratch in a
// file-scope device array instead of a caller workspace.
#include <mutex>

#include "common.h"

namespace adept {
namespace {

constexpr int kTileM = 256;
constexpr int kMaxLayers = 1024;

struct KvWs {
  int32_t* n_work;
  int32_t* grp_m;
  int32_t* work;
  int32_t* srows;
  float* rinv;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

KvWs carve(void* ws, int n_layers, int max_rows, size_t* total) {
  char* p = (char*)ws;
  size_t off = 0;
  KvWs w{};
  w.n_work = (int32_t*)(p + off); off += 256;
  w.grp_m = (int32_t*)(p + off); off += align256((size_t)(n_layers + 2) * 4);
  const size_t max_work = (size_t)n_layers * ((max_rows + kTileM - 1) / kTileM);
  w.work = (int32_t*)(p + off); off += align256(max_work * 4);
  w.srows = (int32_t*)(p + off); off += align256((size_t)max_rows * 4);
  w.rinv = (float*)(p + off); off += align256((size_t)max_rows * 4);
  *total = off;
  return w;
}

__global__ __launch_bounds__(1024) void kv_plan_kernel(int n_layers, const int32_t* __restrict__ rows,
                                                       const int32_t* __restrict__ n_rows,
                                                       int max_rows,
                                                       const int32_t* __restrict__ exit_layer,
                                                       KvWs w) {
  __shared__ int hist[kMaxLayers + 2];
  __shared__ int cursor[kMaxLayers + 2];
  const int n = min(*n_rows, max_rows);
  for (int l = threadIdx.x; l <= n_layers + 1; l += blockDim.x) hist[l] = 0;
  __syncthreads();
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    int L = exit_layer[rows[k]];
    L = L < 0 ? 0 : (L > n_layers ? n_layers : L);
    atomicAdd(&hist[L], 1);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // grp_m[r] = rows with exit layer < r; cursor[L] = first sorted slot of bin L
    int run = 0;
    for (int L = 0; L <= n_layers; ++L) {
      w.grp_m[L] = run;
      cursor[L] = run;
      run += hist[L];
    }
    w.grp_m[n_layers + 1] = run;
    int nw = 0;
    for (int r = 1; r <= n_layers; ++r) {
      const int tiles = (w.grp_m[r] + kTileM - 1) / kTileM;
      for (int t = 0; t < tiles; ++t) w.work[nw++] = (r << 16) | t;
    }
    *w.n_work = nw;
  }
  __syncthreads();
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    const int row = rows[k];
    int L = exit_layer[row];
    L = L < 0 ? 0 : (L > n_layers ? n_layers : L);
    const int at = atomicAdd(&cursor[L], 1);
    w.srows[at] = row;
  }
}

__global__ __launch_bounds__(256) void kv_rinv_kernel(int d, float eps, const bf16* __restrict__ s,
                                                      const int32_t* __restrict__ n_rows,
                                                      int max_rows, KvWs w) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= min(*n_rows, max_rows)) return;
  const bf16* x = s + (int64_t)w.srows[m] * d;
  float ss = 0.0f;
  for (int c = lane * 8; c < d; c += 64 * 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(x + c);
    const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
      ss = fmaf(lo, lo, ss);
      ss = fmaf(hi, hi, ss);
    }
  }
  ss = wave_sum_f32(ss);
  if (lane == 0) w.rinv[m] = 1.0f / sqrtf(ss / (float)d + eps);
}

__global__ __launch_bounds__(256) void kvgen_f32_kernel(
    int n_layers, int d, int H, int hd, float eps, const float* __restrict__ s,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ n_rows, int max_rows,
    const int32_t* __restrict__ exit_layer, const int32_t* __restrict__ slot,
    const int32_t* __restrict__ pos, const float* __restrict__ w_kv, int64_t w_stride,
    const float* __restrict__ gain, const float* __restrict__ rc, const float* __restrict__ rsn,
    float* __restrict__ kc, float* __restrict__ vc, int64_t layer_stride) {
  extern __shared__ float ksm[];
  float* u = ksm;          // [d]
  float* kraw = ksm + d;   // [H*hd]
  __shared__ float red[4];
  const int k = blockIdx.x, r = blockIdx.y + 1, tid = threadIdx.x;
  if (k >= min(*n_rows, max_rows)) return;
  const int row = rows[k];
  if (r <= exit_layer[row]) return;
  const float* x = s + (int64_t)row * d;
  float ss = 0.0f;
  for (int c = tid; c < d; c += 256) ss = fmaf(x[c], x[c], ss);
  ss = wave_sum_f32(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float rinv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
  const float* g = gain ? gain + (int64_t)(r - 1) * d : nullptr;
  for (int c = tid; c < d; c += 256) u[c] = x[c] * rinv * (g ? g[c] : 1.0f);
  __syncthreads();
  const int dq = H * hd;
  const float* W = w_kv + (int64_t)(r - 1) * w_stride;
  const int64_t dst = (int64_t)(r - 1) * layer_stride + (int64_t)slot[row] * dq;
  for (int o = tid; o < 2 * dq; o += 256) {
    const float* wr = W + (int64_t)o * d;
    float a = 0.0f;
    for (int c = 0; c < d; ++c) a = fmaf(u[c], wr[c], a);
    if (o < dq) kraw[o] = a;
    else vc[dst + o - dq] = a;
  }
  __syncthreads();
  const int half = hd / 2, p = pos[row];
  for (int o = tid; o < dq; o += 256) {
    const int c = o % hd, kk = c % half;
    const float cs = rc[(int64_t)p * half + kk], sn = rsn[(int64_t)p * half + kk];
    const float xv = kraw[o], y = c < half ? kraw[o + half] : kraw[o - half];
    kc[dst + o] = c < half ? xv * cs - y * sn : xv * cs + y * sn;
  }
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_kv_generate_workspace_bytes(int n_layers, int max_rows) {
  size_t total = 0;
  carve(nullptr, n_layers, max_rows, &total);
  return total;
}

extern "C" adept_status adept_kv_generate(adept_dtype dt, int n_layers, int d_model, int n_heads,
                                          int head_dim, float eps, const void* s_map,
                                          const int32_t* rows, const int32_t* n_rows,
                                          int max_rows, const int32_t* exit_layer,
                                          const int32_t* cache_slot, const int32_t* pos,
                                          const void* w_kv, int64_t w_kv_layer_stride,
                                          const void* attn_gain, const float* rope_cos,
                                          const float* rope_sin, int rope_max_pos,
                                          void* k_cache, void* v_cache, int64_t n_slots,
                                          void* workspace, size_t workspace_bytes,
                                          void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "kv_generate: bad dtype");
  ADEPT_REQUIRE(n_layers >= 1 && n_layers <= kMaxLayers, "kv_generate: n_layers %d", n_layers);
  ADEPT_REQUIRE(d_model > 0 && n_heads > 0 && head_dim > 0 && head_dim % 2 == 0,
                "kv_generate: bad sizes");
  ADEPT_REQUIRE(max_rows >= 0 && n_slots > 0 && rope_max_pos > 0, "kv_generate: bad sizes");
  ADEPT_REQUIRE(max_rows < (1 << 24), "kv_generate: max_rows too large");
  ADEPT_REQUIRE(s_map && rows && n_rows && exit_layer && cache_slot && pos && w_kv && rope_cos &&
                    rope_sin && k_cache && v_cache,
                "kv_generate: NULL tensor");
  ADEPT_REQUIRE(dt == ADEPT_F32 || attn_gain == nullptr,
                "kv_generate: bf16 takes the gains folded into w_kv (adept_fold_gain); "
                "pass attn_gain = NULL");
  const int dq = n_heads * head_dim;
  ADEPT_REQUIRE(w_kv_layer_stride >= (int64_t)2 * dq * d_model,
                "kv_generate: layer stride %lld below 2*H*hd*D", (long long)w_kv_layer_stride);
  if (max_rows == 0) return ADEPT_OK;
  hipStream_t s = as_stream(stream);
  const int64_t layer_stride = n_slots * dq;
  if (dt == ADEPT_F32) {
    ADEPT_REQUIRE(d_model <= 8192 && dq <= 8192, "kv_generate: f32 path limited to width 8192");
    const size_t smem = (size_t)(d_model + dq) * sizeof(float);
    ADEPT_LAUNCH(kvgen_f32_kernel, dim3(max_rows, n_layers), dim3(256), smem, s, n_layers,
                       d_model, n_heads, head_dim, eps, (const float*)s_map, rows, n_rows,
                       max_rows, exit_layer, cache_slot, pos, (const float*)w_kv,
                       w_kv_layer_stride, (const float*)attn_gain, rope_cos, rope_sin,
                       (float*)k_cache, (float*)v_cache, layer_stride);
    return launch_status("kvgen_f32");
  }
  ADEPT_REQUIRE(d_model % 64 == 0, "kv_generate: bf16 needs d_model %% 64 == 0");
  ADEPT_REQUIRE((head_dim == 64 || head_dim == 128) && dq % 256 == 0,
                "kv_generate: bf16 needs head_dim 64/128 and H*hd %% 256 == 0");
  ADEPT_REQUIRE(aligned16(s_map) && aligned16(w_kv) && aligned16(workspace) &&
                    w_kv_layer_stride % 8 == 0,
                "kv_generate: tensors must be 16-byte aligned");
  size_t need = 0;
  carve(nullptr, n_layers, max_rows, &need);
  if (!workspace || workspace_bytes < need) {
    set_error("kv_generate: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  KvWs w = carve(workspace, n_layers, max_rows, &need);
  ADEPT_LAUNCH(kv_plan_kernel, dim3(1), dim3(1024), 0, s, n_layers, rows, n_rows, max_rows,
                     exit_layer, w);
  ADEPT_CHECK_LAUNCH("kv_plan");
  ADEPT_LAUNCH(kv_rinv_kernel, dim3(ceil_div(max_rows, 4)), dim3(256), 0, s, d_model, eps,
                     (const bf16*)s_map, n_rows, max_rows, w);
  ADEPT_CHECK_LAUNCH("kv_rinv");
  GemmArgs g{};
  g.M_max = max_rows; g.N = 2 * dq; g.K = d_model;
  g.A = s_map; g.lda = d_model; g.B = w_kv; g.ldb = d_model;
  g.epi = EPI_KV; g.pos = pos; g.slot = cache_slot;
  g.rope_cos = rope_cos; g.rope_sin = rope_sin; g.head_dim = head_dim; g.d_q = dq;
  g.k_cache = k_cache; g.v_cache = v_cache; g.row_scale = w.rinv;
  const int max_work = n_layers * ceil_div(max_rows, kTileM);
  return gemm_kv_grouped(g, w.work, w.n_work, max_work, w.grp_m, w.srows,
                         w_kv_layer_stride, layer_stride, s);
}

// ---------------------------------------------------------------------------
// LayerNorm family (GPT-2 style): s~ is normalised once, without the affine
// part (the same for every skipped layer); layer r's LayerNorm gain is folded
// into the columns of its Wk / Wv and its shift into their biases
// (adept_fold_gain, adept_fold_bias), so the grouped GEMM takes the
// normalised rows (in sorted order) and adds layer r's bias; no RoPE.
// ---------------------------------------------------------------------------
namespace adept {
namespace {

size_t ln_total(int n_layers, int max_rows, int d_model, size_t* xhat_off) {
  size_t base = 0;
  carve(nullptr, n_layers, max_rows, &base);
  *xhat_off = base;
  return base + align256((size_t)max_rows * d_model * 2);
}

}  // namespace
}  // namespace adept

extern "C" size_t adept_kv_generate_layernorm_workspace_bytes(int n_layers, int max_rows,
                                                              int d_model) {
  size_t off = 0;
  return ln_total(n_layers, max_rows, d_model, &off);
}

extern "C" adept_status adept_kv_generate_layernorm(
    adept_dtype dt, int n_layers, int d_model, int n_heads, int head_dim, float eps,
    const void* s_map, const int32_t* rows, const int32_t* n_rows, int max_rows,
    const int32_t* exit_layer, const int32_t* cache_slot, const void* w_kv,
    int64_t w_kv_layer_stride, const void* b_kv, int64_t b_kv_layer_stride, void* k_cache,
    void* v_cache, int64_t n_slots, void* workspace, size_t workspace_bytes, void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_BF16, "kv_generate_layernorm: bf16 only");
  ADEPT_REQUIRE(n_layers >= 1 && n_layers <= kMaxLayers, "kv_generate_layernorm: n_layers %d",
                n_layers);
  ADEPT_REQUIRE(d_model > 0 && d_model % 64 == 0 && n_heads > 0 && head_dim > 0,
                "kv_generate_layernorm: d_model must be a multiple of 64");
  const int dq = n_heads * head_dim;
  ADEPT_REQUIRE(dq % 32 == 0, "kv_generate_layernorm: H*hd must be a multiple of 32");
  ADEPT_REQUIRE(max_rows >= 0 && max_rows < (1 << 24) && n_slots > 0,
                "kv_generate_layernorm: bad sizes");
  ADEPT_REQUIRE(s_map && rows && n_rows && exit_layer && cache_slot && w_kv && b_kv && k_cache &&
                    v_cache,
                "kv_generate_layernorm: NULL tensor");
  ADEPT_REQUIRE(w_kv_layer_stride >= (int64_t)2 * dq * d_model && w_kv_layer_stride % 8 == 0 &&
                    b_kv_layer_stride >= 2 * dq && b_kv_layer_stride % 4 == 0,
                "kv_generate_layernorm: layer strides");
  ADEPT_REQUIRE(aligned16(s_map) && aligned16(w_kv) && aligned16(workspace) &&
                    ((uintptr_t)b_kv & 7) == 0,
                "kv_generate_layernorm: tensors must be 16-byte aligned (bias 8)");
  if (max_rows == 0) return ADEPT_OK;
  size_t xoff = 0;
  const size_t need = ln_total(n_layers, max_rows, d_model, &xoff);
  if (!workspace || workspace_bytes < need) {
    set_error("kv_generate_layernorm: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  hipStream_t s = as_stream(stream);
  size_t tmp = 0;
  KvWs w = carve(workspace, n_layers, max_rows, &tmp);
  void* xhat = (char*)workspace + xoff;
  ADEPT_LAUNCH(kv_plan_kernel, dim3(1), dim3(1024), 0, s, n_layers, rows, n_rows, max_rows,
               exit_layer, w);
  ADEPT_CHECK_LAUNCH("kv_plan");
  // the exited rows, normalised in sorted order
  ADEPT_TRY(layernorm_rows_sel(dt, d_model, eps, s_map, s_map, nullptr, w.srows, n_rows, max_rows,
                               nullptr, nullptr, xhat, s));
  GemmArgs g{};
  g.M_max = max_rows; g.N = 2 * dq; g.K = d_model;
  g.A = xhat; g.lda = d_model; g.a_sorted = 1; g.B = w_kv; g.ldb = d_model;
  g.epi = EPI_KV; g.slot = cache_slot; g.head_dim = head_dim; g.d_q = dq;
  g.k_cache = k_cache; g.v_cache = v_cache;
  g.bias = b_kv; g.bias_layer_stride = b_kv_layer_stride;
  const int max_work = n_layers * ceil_div(max_rows, kTileM);
  return gemm_kv_grouped(g, w.work, w.n_work, max_work, w.grp_m, w.srows,
                         w_kv_layer_stride, n_slots * dq, s);
}

// ---------------------------------------------------------------------------
// Allocation-free variant: the plan / work-list / row-scale scratch lives in
// a file-scope device array (one copy per GPU, kept until the process ends).
// Host code never passes the array's name to a kernel: its device address is
// looked up once per device with hipGetSymbolAddress and kept per device.
// ---------------------------------------------------------------------------
namespace adept {
namespace {

constexpr size_t kNoallocScratchBytes = (size_t)4 << 20;
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array's device address on the current device (looked up on
// the first call made with that device current); nullptr with the error set.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("kv_generate_noalloc: no usable current device (%d)", dev);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      set_error("kv_generate_noalloc: hipGetSymbolAddress failed on device %d: %s", dev,
                hipGetErrorString(e));
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace adept

extern "C" adept_status adept_kv_generate_noalloc(
    adept_dtype dt, int n_layers, int d_model, int n_heads, int head_dim, float eps,
    const void* s_map, const int32_t* rows, const int32_t* n_rows, int max_rows,
    const int32_t* exit_layer, const int32_t* cache_slot, const int32_t* pos, const void* w_kv,
    int64_t w_kv_layer_stride, const void* attn_gain, const float* rope_cos,
    const float* rope_sin, int rope_max_pos, void* k_cache, void* v_cache, int64_t n_slots,
    void* stream) {
  ADEPT_REQUIRE(n_layers >= 1 && n_layers <= kMaxLayers && max_rows >= 0 &&
                    max_rows < (1 << 24),
                "kv_generate_noalloc: bad sizes");
  size_t need = 0;
  carve(nullptr, n_layers, max_rows, &need);
  if (need > kNoallocScratchBytes) {
    set_error("kv_generate_noalloc: %d layers x %d rows need %zu bytes of scratch, above the "
              "fixed %zu; use adept_kv_generate with a workspace",
              n_layers, max_rows, need, kNoallocScratchBytes);
    return ADEPT_E_UNSUPPORTED;
  }
  void* ws = scratch_on_current_device();
  if (!ws) return ADEPT_E_HIP;
  return adept_kv_generate(dt, n_layers, d_model, n_heads, head_dim, eps, s_map, rows, n_rows,
                           max_rows, exit_layer, cache_slot, pos, w_kv, w_kv_layer_stride,
                           attn_gain, rope_cos, rope_sin, rope_max_pos, k_cache, v_cache, n_slots,
                           ws, kNoallocScratchBytes, stream);
}
