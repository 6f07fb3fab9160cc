// Dense and grouped GEMMs of the hot path, C[m][n] = sum_k A[m][k] B[n][k]
// (B in nn.Linear [out][in] order, so both operands are K-contiguous).
//
// bf16 path: one 256-thread workgroup computes a 256x256 output tile with
// v_mfma_f32_32x32x16_bf16; its four waves each own a 128x128 sub-tile
// (4x4 MFMA blocks, 256 accumulators per lane).  K advances 64 at a time
// through a double-buffered LDS stage (rows padded to 72 elements so the
// 16-byte MFMA operand reads are conflict-free); the next stage's global
// loads are issued before the current stage's MFMAs so HBM latency hides
// behind matrix work, and one barrier per stage orders the buffer swap.
//
// Epilogues run on the accumulators in registers.  A 128-column wave
// sub-tile covers whole heads (head_dim 64 or 128), so the rotary pair
// (c, c + hd/2) of a column sits in the same lane (block nb ^ hd/64) and
// RoPE is applied there before K/V are stored into their cache slots.
//
// The grouped variant is the decoupled KV generation of Eq. 9: work items
// (layer r, 256-row tile) come from a device-built list over the exited rows
// sorted by exit layer, so the rows with i* < r are a prefix; A is formed
// while staging as bf16(s~ * rsqrt(mean s~^2 + eps) * gain_r), B is
// [Wk_r; Wv_r], and the epilogue writes K (with RoPE) and V to cache[r].
//
// f32 path (small configurations only): a plain 64x64-tiled FMA GEMM into a
// float scratch buffer followed by an element-wise epilogue kernel.
#include <algorithm>

#include "common.h"

namespace adept {
namespace {

constexpr int BM = 256, BN = 256, BK = 64, LDK = BK + 8;
constexpr int kThreads = 256;
constexpr size_t kLdsBytes = (size_t)2 * (BM + BN) * LDK * sizeof(bf16);  // 147456
constexpr int kPersistentBlocks = 256;  // one workgroup per CU (LDS-limited)

struct GP {
  int M_max;
  const int32_t* M_dev;
  int N, K;
  const bf16* A;
  const int32_t* a_rows;
  int64_t lda;
  const bf16* B;
  const bf16* B2;
  int64_t ldb;
  void* C;
  int64_t ldc;
  int c_f32;
  const int32_t* rows;
  const bf16* resid;
  const int32_t* pos;
  const int32_t* slot;
  const float* rope_cos;
  const float* rope_sin;
  int head_dim, d_q;
  bf16* q_out;
  bf16* k_cache;
  bf16* v_cache;
  // grouped (KV generation)
  const int32_t* work;      // packed (layer << 16) | m_tile
  const int32_t* n_work;
  const int32_t* grp_m;     // [N+2]: rows with exit layer < r
  const int32_t* srows;     // exited rows sorted by exit layer
  const float* rinv;        // [sorted index] 1/sqrt(mean s^2 + eps)
  const bf16* gain;         // [N][K]
  int64_t b_layer_stride;
  int64_t cache_layer_stride;
  int n_tiles_n;
};

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// One 256x256 output tile: rows [mt*256, M) of A against B tile nt.
template <int EPI, bool GROUPED>
__device__ __forceinline__ void gemm_tile(const GP& p, bf16* smem, int layer, int mt, int nt,
                                          int M, const bf16* Bm) {
  bf16* sA = smem;
  bf16* sB = smem + 2 * BM * LDK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = mt * BM;

  // ---- per-thread load assignments: 8 rows (r0 + 32 j) x one 16-byte chunk
  const int lr0 = tid >> 3, lc = (tid & 7) * 8;
  const bf16* a_src[8];
  const bf16* b_src[8];
  float a_scale[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = lr0 + 32 * j;
    int m = m0 + r;
    if (m >= M) m = m0;  // clamp: loaded but never stored
    int arow;
    if (GROUPED) {
      arow = p.srows[m];
      a_scale[j] = p.rinv[m];
    } else {
      arow = p.a_rows ? p.a_rows[m] : m;
      a_scale[j] = 1.0f;
    }
    a_src[j] = p.A + (int64_t)arow * p.lda + lc;
    int64_t brow;
    const bf16* bbase = Bm;
    if (EPI == EPI_SWIGLU) {
      const int half = r >> 7, within = r & 127;
      bbase = within < 64 ? p.B : p.B2;
      brow = (int64_t)nt * 128 + half * 64 + (within & 63);
    } else {
      brow = (int64_t)nt * BN + r;
    }
    b_src[j] = bbase + brow * p.ldb + lc;
  }
  const bf16* gain_src = GROUPED ? p.gain + (int64_t)(layer - 1) * p.K + lc : nullptr;

  uint4 ra[8], rb[8];
  auto load_stage = [&](int k0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      ra[j] = *reinterpret_cast<const uint4*>(a_src[j] + k0);
      rb[j] = *reinterpret_cast<const uint4*>(b_src[j] + k0);
    }
  };
  auto store_stage = [&](int buf, int k0) {
    bf16* dA = sA + buf * BM * LDK;
    bf16* dB = sB + buf * BN * LDK;
    if (GROUPED) {
      const uint4 gv = *reinterpret_cast<const uint4*>(gain_src + k0);
      const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
      float g[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        g[2 * e] = __uint_as_float(gw[e] << 16);
        g[2 * e + 1] = __uint_as_float(gw[e] & 0xffff0000u);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t w[4] = {ra[j].x, ra[j].y, ra[j].z, ra[j].w};
        uint32_t o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(w[e] << 16) * a_scale[j] * g[2 * e];
          const float hi = __uint_as_float(w[e] & 0xffff0000u) * a_scale[j] * g[2 * e + 1];
          o[e] = (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
        }
        ra[j] = make_uint4(o[0], o[1], o[2], o[3]);
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int r = lr0 + 32 * j;
      *reinterpret_cast<uint4*>(dA + r * LDK + lc) = ra[j];
      *reinterpret_cast<uint4*>(dB + r * LDK + lc) = rb[j];
    }
  };

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  const int KT = p.K / BK;
  load_stage(0);
  store_stage(0, 0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_stage((kt + 1) * BK);
    const bf16* cA = sA + buf * BM * LDK + (wm * 128 + (lane & 31)) * LDK + (lane >> 5) * 8;
    const bf16* cB = sB + buf * BN * LDK + (wn * 128 + (lane & 31)) * LDK + (lane >> 5) * 8;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8_t a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = *reinterpret_cast<const bf16x8_t*>(cA + i * 32 * LDK + ks * 16);
        b[i] = *reinterpret_cast<const bf16x8_t*>(cB + i * 32 * LDK + ks * 16);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) store_stage(buf ^ 1, (kt + 1) * BK);
    __syncthreads();
  }

  // ---- epilogues.  Lane holds column (lane & 31) of each 32x32 block and
  // rows 8*(v/4) + 4*(lane/32) + v%4, v = 0..15.
  const int col_l = lane & 31;
  const int row_q = 4 * (lane >> 5);
  if (EPI == EPI_STORE || EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm * 128 + i * 32 + 8 * (v >> 2) + row_q + (v & 3);
        if (m >= M) continue;
        const int64_t orow = EPI == EPI_RESID ? (int64_t)p.rows[m] : (int64_t)m;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = nt * BN + wn * 128 + j * 32 + col_l;
          float x = acc[i][j][v];
          if (EPI == EPI_RESID) {
            x += bf2f(p.resid[orow * p.ldc + n]);
            reinterpret_cast<bf16*>(p.C)[orow * p.ldc + n] = f2bf(x);
          } else if (p.c_f32) {
            reinterpret_cast<float*>(p.C)[orow * p.ldc + n] = x;
          } else {
            reinterpret_cast<bf16*>(p.C)[orow * p.ldc + n] = f2bf(x);
          }
        }
      }
  } else if (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm * 128 + i * 32 + 8 * (v >> 2) + row_q + (v & 3);
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int o = nt * 128 + wn * 64 + j * 32 + col_l;
          const float g = acc[i][j][v], u = acc[i][j + 2][v];
          reinterpret_cast<bf16*>(p.C)[(int64_t)m * p.ldc + o] = f2bf(silu(g) * u);
        }
      }
  } else {  // EPI_QKV / EPI_KV
    const int nw = nt * BN + wn * 128;          // first output column of this wave
    const int sec = nw / p.d_q;                 // QKV: 0 q, 1 k, 2 v;  KV: 0 k, 1 v
    const bool is_q = EPI == EPI_QKV && sec == 0;
    const bool is_v = EPI == EPI_QKV ? sec == 2 : sec == 1;
    const int cbase = nw - sec * p.d_q;         // column within the section
    const int hd = p.head_dim, half = hd >> 1, pmask = hd >> 6;
    bf16* kc = p.k_cache;
    bf16* vc = p.v_cache;
    if (GROUPED) {
      kc += (int64_t)(layer - 1) * p.cache_layer_stride;
      vc += (int64_t)(layer - 1) * p.cache_layer_stride;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm * 128 + i * 32 + 8 * (v >> 2) + row_q + (v & 3);
        if (m >= M) continue;
        const int row = GROUPED ? p.srows[m] : p.rows[m];
        bf16* dst;
        if (is_q) dst = p.q_out + (int64_t)m * p.d_q;
        else dst = (is_v ? vc : kc) + (int64_t)p.slot[row] * p.d_q;
        if (is_v) {
#pragma unroll
          for (int j = 0; j < 4; ++j) dst[cbase + j * 32 + col_l] = f2bf(acc[i][j][v]);
        } else {
          const int ps = p.pos[row];
          const float* cr = p.rope_cos + (int64_t)ps * half;
          const float* sr = p.rope_sin + (int64_t)ps * half;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int c = (cbase + j * 32 + col_l) % hd;  // column within the head
            const int kk = c % half;
            const float cs = cr[kk], sn = sr[kk];
            const float x = acc[i][j][v];
            const float y = acc[i][j ^ pmask][v];          // partner column c +- hd/2
            const float r = c < half ? x * cs - y * sn : x * cs + y * sn;
            dst[cbase + j * 32 + col_l] = f2bf(r);
          }
        }
      }
  }
}

template <int EPI>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(GP p) {
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  const int M = p.M_dev ? min(*p.M_dev, p.M_max) : p.M_max;
  if ((int)blockIdx.x * BM >= M) return;
  gemm_tile<EPI, false>(p, smem, 0, blockIdx.x, blockIdx.y, M, p.B);
}

// Persistent grouped GEMM: workgroups stride over the device-built list of
// (layer, row tile) items times the column tiles; an empty list costs one
// read per workgroup.
__global__ __launch_bounds__(kThreads, 1) void gemm_kv_grouped_kernel(GP p) {
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  const int total = *p.n_work * p.n_tiles_n;
  for (int item = blockIdx.x; item < total; item += gridDim.x) {
    const int w = item / p.n_tiles_n, nt = item % p.n_tiles_n;
    const int packed = p.work[w];
    const int layer = packed >> 16, mt = packed & 0xffff;
    const int M = p.grp_m[layer];
    gemm_tile<EPI_KV, true>(p, smem, layer, mt, nt, M,
                            p.B + (int64_t)(layer - 1) * p.b_layer_stride);
    __syncthreads();  // LDS is reused by the next item
  }
}

// ----------------------------------------------------------------------------
// f32 path
// ----------------------------------------------------------------------------
constexpr int FT = 64, FK = 16;

__global__ __launch_bounds__(256) void gemm_f32_kernel(int M_max, const int32_t* M_dev, int N,
                                                       int K, const float* __restrict__ A,
                                                       const int32_t* __restrict__ a_rows,
                                                       int64_t lda, const float* __restrict__ B,
                                                       int64_t ldb, float* __restrict__ C,
                                                       int64_t ldc) {
  __shared__ float sA[FK][FT + 1];
  __shared__ float sB[FK][FT + 1];
  const int M = M_dev ? min(*M_dev, M_max) : M_max;
  const int m0 = blockIdx.x * FT, n0 = blockIdx.y * FT;
  if (m0 >= M) return;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FK) {
    for (int e = threadIdx.x; e < FT * FK; e += 256) {
      const int r = e / FK, c = e % FK;
      int m = m0 + r;
      const bool mv = m < M;
      if (!mv) m = m0;
      const int arow = a_rows ? a_rows[m] : m;
      sA[c][r] = (k0 + c < K) ? A[(int64_t)arow * lda + k0 + c] : 0.0f;
      const int n = n0 + r;
      sB[c][r] = (n < N && k0 + c < K) ? B[(int64_t)n * ldb + k0 + c] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < FK; ++c) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[c][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[c][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < N) C[(int64_t)m * ldc + n] = acc[i][j];
    }
  }
}

// Element-wise epilogue over the f32 scratch T[m][n] (n < n_out).
__global__ void epilogue_f32_kernel(int epi, int M_max, const int32_t* M_dev, int n_out,
                                    const float* __restrict__ T, int64_t ldt, GP p) {
  const int M = M_dev ? min(*M_dev, M_max) : M_max;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int m = (int)(idx / n_out), n = (int)(idx % n_out);
  if (m >= M) return;
  const float* t = T + (int64_t)m * ldt;
  float* C = reinterpret_cast<float*>(p.C);
  if (epi == EPI_STORE) {
    C[(int64_t)m * p.ldc + n] = t[n];
  } else if (epi == EPI_RESID) {
    const int64_t row = p.rows[m];
    C[row * p.ldc + n] = reinterpret_cast<const float*>(p.resid)[row * p.ldc + n] + t[n];
  } else if (epi == EPI_SWIGLU) {
    C[(int64_t)m * p.ldc + n] = silu(t[n]) * t[p.N + n];
  } else {  // EPI_QKV
    const int sec = n / p.d_q, cin = n - sec * p.d_q;
    const int row = p.rows[m];
    float* dst;
    if (sec == 0) dst = reinterpret_cast<float*>(p.q_out) + (int64_t)m * p.d_q;
    else dst = reinterpret_cast<float*>(sec == 1 ? p.k_cache : p.v_cache) + (int64_t)p.slot[row] * p.d_q;
    if (sec == 2) {
      dst[cin] = t[n];
    } else {
      const int hd = p.head_dim, half = hd / 2;
      const int c = cin % hd, kk = c % half;
      const int ps = p.pos[row];
      const float cs = p.rope_cos[(int64_t)ps * half + kk], sn = p.rope_sin[(int64_t)ps * half + kk];
      const float x = t[n];
      const float y = c < half ? t[n + half] : t[n - half];
      dst[cin] = c < half ? x * cs - y * sn : x * cs + y * sn;
    }
  }
}

template <int EPI>
adept_status launch_bf16(const GP& p, dim3 grid, hipStream_t s, const char* name) {
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute((const void*)gemm_bf16_kernel<EPI>,
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kLdsBytes) != hipSuccess)
      return launch_status("gemm_bf16 LDS attribute");
    attr_set = true;
  }
  {
    TimedLaunch tl(name ? name : "gemm_bf16", s);
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI>), grid, dim3(kThreads), kLdsBytes, s, p);
  }
  return launch_status("gemm_bf16");
}

GP to_gp(const GemmArgs& g) {
  GP p{};
  p.M_max = g.M_max; p.M_dev = g.M_dev; p.N = g.N; p.K = g.K;
  p.A = (const bf16*)g.A; p.a_rows = g.a_rows; p.lda = g.lda;
  p.B = (const bf16*)g.B; p.B2 = (const bf16*)g.B2; p.ldb = g.ldb;
  p.C = g.C; p.ldc = g.ldc; p.c_f32 = g.c_f32;
  p.rows = g.rows; p.resid = (const bf16*)g.resid; p.pos = g.pos; p.slot = g.slot;
  p.rope_cos = g.rope_cos; p.rope_sin = g.rope_sin; p.head_dim = g.head_dim; p.d_q = g.d_q;
  p.q_out = (bf16*)g.q_out; p.k_cache = (bf16*)g.k_cache; p.v_cache = (bf16*)g.v_cache;
  return p;
}

}  // namespace

adept_status gemm(adept_dtype dt, const GemmArgs& g, hipStream_t s) {
  if (g.M_max <= 0) return ADEPT_OK;
  if (dt == ADEPT_BF16) {
    if (g.K % BK != 0) {
      set_error("gemm: K=%d not a multiple of %d", g.K, BK);
      return ADEPT_E_UNSUPPORTED;
    }
    const int ncols = g.epi == EPI_SWIGLU ? 128 : BN;
    if (g.N % ncols != 0) {
      set_error("gemm: N=%d not a multiple of %d", g.N, ncols);
      return ADEPT_E_UNSUPPORTED;
    }
    if ((g.epi == EPI_QKV) && (g.d_q % 128 != 0 || (g.head_dim != 64 && g.head_dim != 128))) {
      set_error("gemm: QKV epilogue needs head_dim 64/128 and d_q %% 128 == 0");
      return ADEPT_E_UNSUPPORTED;
    }
    GP p = to_gp(g);
    dim3 grid(ceil_div(g.M_max, BM), g.N / ncols);
    switch (g.epi) {
      case EPI_STORE: return launch_bf16<EPI_STORE>(p, grid, s, g.name);
      case EPI_QKV: return launch_bf16<EPI_QKV>(p, grid, s, g.name);
      case EPI_RESID: return launch_bf16<EPI_RESID>(p, grid, s, g.name);
      case EPI_SWIGLU: return launch_bf16<EPI_SWIGLU>(p, grid, s, g.name);
      default: set_error("gemm: bad epilogue"); return ADEPT_E_INVALID;
    }
  }
  // f32: scratch T[M_max][n_t] in g.tmp (passed through C when epi == STORE)
  set_error("gemm: f32 path needs gemm_f32()");
  return ADEPT_E_INVALID;
}

// f32 GEMM + element-wise epilogue; tmp holds M_max x (N or 2N for SWIGLU) floats.
adept_status gemm_f32(const GemmArgs& g, float* tmp, hipStream_t s) {
  if (g.M_max <= 0) return ADEPT_OK;
  const int nt = g.epi == EPI_SWIGLU ? 2 * g.N : g.N;
  dim3 block(256);
  dim3 grid(ceil_div(g.M_max, FT), ceil_div(g.N, FT));
  ADEPT_LAUNCH(gemm_f32_kernel, grid, block, 0, s, g.M_max, g.M_dev, g.N, g.K,
                     (const float*)g.A, g.a_rows, g.lda, (const float*)g.B, g.ldb, tmp,
                     (int64_t)nt);
  ADEPT_CHECK_LAUNCH("gemm_f32");
  if (g.epi == EPI_SWIGLU) {
    ADEPT_LAUNCH(gemm_f32_kernel, grid, block, 0, s, g.M_max, g.M_dev, g.N, g.K,
                       (const float*)g.A, g.a_rows, g.lda, (const float*)g.B2, g.ldb,
                       tmp + g.N, (int64_t)nt);
    ADEPT_CHECK_LAUNCH("gemm_f32");
  }
  GP p = to_gp(g);
  const int64_t total = (int64_t)g.M_max * g.N;
  ADEPT_LAUNCH(epilogue_f32_kernel, dim3((unsigned)((total + 255) / 256)), block, 0, s,
                     g.epi, g.M_max, g.M_dev, g.N, (const float*)tmp, (int64_t)nt, p);
  return launch_status("epilogue_f32");
}

// f32 GEMM written straight to C (no epilogue): C[m][n] = A[m] . B[n].
adept_status gemm_f32_direct(const GemmArgs& g, hipStream_t s) {
  if (g.M_max <= 0) return ADEPT_OK;
  dim3 grid(ceil_div(g.M_max, FT), ceil_div(g.N, FT));
  ADEPT_LAUNCH(gemm_f32_kernel, grid, dim3(256), 0, s, g.M_max, g.M_dev, g.N, g.K,
                     (const float*)g.A, g.a_rows, g.lda, (const float*)g.B, g.ldb,
                     (float*)g.C, g.ldc);
  return launch_status("gemm_f32");
}

// Grouped bf16 GEMM of the KV generation (see the header comment).
adept_status gemm_kv_grouped(const GemmArgs& g, const int32_t* work, const int32_t* n_work,
                             int max_work, const int32_t* grp_m, const int32_t* srows,
                             const float* rinv, const void* gain, int64_t b_layer_stride,
                             int64_t cache_layer_stride, hipStream_t s) {
  if (max_work <= 0) return ADEPT_OK;
  GP p = to_gp(g);
  p.work = work; p.n_work = n_work; p.grp_m = grp_m; p.srows = srows; p.rinv = rinv;
  p.gain = (const bf16*)gain; p.b_layer_stride = b_layer_stride;
  p.cache_layer_stride = cache_layer_stride;
  p.n_tiles_n = g.N / BN;
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute((const void*)gemm_kv_grouped_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kLdsBytes) != hipSuccess)
      return launch_status("gemm_kv_grouped LDS attribute");
    attr_set = true;
  }
  const int grid = std::min(max_work * p.n_tiles_n, kPersistentBlocks);
  ADEPT_LAUNCH(gemm_kv_grouped_kernel, dim3(grid), dim3(kThreads), kLdsBytes, s, p);
  return launch_status("gemm_kv_grouped");
}

}  // namespace adept
