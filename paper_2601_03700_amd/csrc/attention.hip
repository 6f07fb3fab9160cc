// Attention of the active tokens over one layer's cache, whose entries were
// either computed by the layer itself (tokens still active) or generated
// from an earlier exit state (Section 3, Eq. 5; Section 4.3).  The kernels do
// not distinguish the two: a generated entry is an ordinary cache row.
//
// Prefill (bf16, head_dim 64/128, causal): a plan kernel cuts the compacted
// query list into tiles of <= 128 consecutive entries of one sequence; a
// 256-thread workgroup takes one (tile, head), each wave two groups of 16
// queries, so every K/V fragment read from LDS feeds two MFMAs.  Key
// blocks of 64 rows are staged in LDS (K row-major, V transposed with packed
// 8-byte writes of 4 keys), and the
// scores are formed transposed, S^T = K Q^T, with v_mfma_f32_16x16x32_bf16 so
// that each lane owns one query column: the online softmax then needs only
// two cross-lane steps for the running max, and the probabilities already sit
// in the B-operand layout of O^T += V^T P^T (the order of keys inside an
// MFMA's reduction is free, so V^T is read in the same key order).
//
// Generic path (f32, decode with one query per sequence, bidirectional
// attention with a live-key mask): one workgroup per (query, head), scores
// for all keys in LDS, exact softmax, then a weighted sum of V rows.
#include "common.h"

namespace adept {
namespace {

// ---------------------------------------------------------------------------
// generic kernel
// ---------------------------------------------------------------------------
constexpr int kGenThreads = 256;

template <typename T>
__global__ __launch_bounds__(kGenThreads) void attend_generic_kernel(
    int H, int hd, float scale, int causal, const T* __restrict__ q,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ n_active, int max_active,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ seq,
    const T* __restrict__ kc, const T* __restrict__ vc, int s_max,
    const int32_t* __restrict__ key_len, const uint8_t* __restrict__ key_live,
    T* __restrict__ out) {
  extern __shared__ float gsm[];
  float* sq = gsm;             // [hd]
  float* sc = gsm + 128;       // [s_max] scores
  __shared__ float red[kGenThreads / 64];
  __shared__ float part[kGenThreads];
  const int k = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  if (k >= min(*n_active, max_active)) return;
  const int row = rows[k];
  const int b = seq[row];
  const int L = causal ? pos[row] + 1 : key_len[b];
  const int64_t base = (int64_t)b * s_max;
  const int64_t rs = (int64_t)H * hd;  // cache row stride
  for (int d = tid; d < hd; d += kGenThreads) sq[d] = ld(q + (int64_t)k * rs + h * hd + d);
  __syncthreads();
  float mx = -INFINITY;
  for (int t = tid; t < L; t += kGenThreads) {
    const T* kr = kc + (base + t) * rs + h * hd;
    float s = 0.0f;
    for (int d = 0; d < hd; ++d) s = fmaf(sq[d], ld(kr + d), s);
    s *= scale;
    if (key_live && !key_live[base + t]) s = -INFINITY;
    sc[t] = s;
    mx = fmaxf(mx, s);
  }
  mx = wave_max_f32(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  mx = red[0];
  for (int w = 1; w < kGenThreads / 64; ++w) mx = fmaxf(mx, red[w]);
  __syncthreads();
  float sum = 0.0f;
  for (int t = tid; t < L; t += kGenThreads) {
    const float e = sc[t] == -INFINITY ? 0.0f : __expf(sc[t] - mx);
    sc[t] = e;
    sum += e;
  }
  sum = wave_sum_f32(sum);
  if ((tid & 63) == 0) red[tid >> 6] = sum;
  __syncthreads();
  sum = 0.0f;
  for (int w = 0; w < kGenThreads / 64; ++w) sum += red[w];
  // o[d] = sum_t p_t v_t[d]: thread handles dim d = tid % hd over keys t = g, g + G, ...
  const int G = kGenThreads / hd;  // hd divides 256
  const int d = tid % hd, g = tid / hd;
  float o = 0.0f;
  for (int t = g; t < L; t += G) o = fmaf(sc[t], ld(vc + (base + t) * rs + h * hd + d), o);
  part[tid] = o;
  __syncthreads();
  if (g == 0) {
    for (int j = 1; j < G; ++j) o += part[j * hd + d];
    st(out + (int64_t)k * rs + h * hd + d, o / sum);
  }
}

// ---------------------------------------------------------------------------
// prefill plan: tiles of <= 64 consecutive query entries of one sequence
// ---------------------------------------------------------------------------
constexpr int QT = 128;  // queries per tile (4 waves x 2 groups of 16)
constexpr int KB = 64;   // keys per LDS block

__global__ __launch_bounds__(1024) void attend_plan_kernel(const int32_t* __restrict__ rows,
                                                           const int32_t* __restrict__ n_active,
                                                           int max_active,
                                                           const int32_t* __restrict__ seq,
                                                           int n_seq, int2* __restrict__ tiles,
                                                           int32_t* __restrict__ n_tiles) {
  extern __shared__ int psm[];   // [n_seq + 1] segment starts, then [n_seq + 1] tile offsets
  int* seg = psm;
  int* toff = psm + n_seq + 1;
  const int n = min(*n_active, max_active);
  for (int b = threadIdx.x; b <= n_seq; b += blockDim.x) {
    // first entry whose sequence is >= b (sequence ids are non-decreasing)
    int lo = 0, hi = n;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (seq[rows[mid]] < b) lo = mid + 1; else hi = mid;
    }
    seg[b] = lo;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int b = 0; b < n_seq; ++b) {
      toff[b] = acc;
      acc += (seg[b + 1] - seg[b] + QT - 1) / QT;
    }
    toff[n_seq] = acc;
    *n_tiles = acc;
  }
  __syncthreads();
  for (int b = 0; b < n_seq; ++b) {
    const int cnt = seg[b + 1] - seg[b];
    const int nt = (cnt + QT - 1) / QT;
    for (int t = threadIdx.x; t < nt; t += blockDim.x)
      tiles[toff[b] + t] = make_int2(seg[b] + t * QT, min(QT, cnt - t * QT));
  }
}

// ---------------------------------------------------------------------------
// prefill MFMA kernel
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(256, 2) void attend_prefill_kernel(
    int H, float scale_log2, const bf16* __restrict__ q, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ seq,
    const bf16* __restrict__ kc, const bf16* __restrict__ vc, int s_max,
    const int2* __restrict__ tiles, const int32_t* __restrict__ n_tiles, bf16* __restrict__ out) {
  constexpr int KLD = HD + 8;     // sK row stride (elements)
  constexpr int VLD = KB + 8;     // sVt row stride
  constexpr int DS = HD / 32;     // 32-wide dim steps for S
  constexpr int DB = HD / 16;     // 16-row dim blocks of O^T
  constexpr int QG = QT / 64;     // 16-query groups per wave
  __shared__ __attribute__((aligned(16))) bf16 sK[KB * KLD];
  __shared__ __attribute__((aligned(16))) bf16 sVt[HD * VLD];
  const int nt = *n_tiles;
  if ((int)blockIdx.x >= nt) return;
  const int2 tile = tiles[nt - 1 - blockIdx.x];   // longest (latest) tiles first
  const int h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int64_t rs = (int64_t)H * HD;

  const int b = seq[rows[tile.x]];
  const int pmax = pos[rows[tile.x + tile.y - 1]];
  const int64_t kbase = (int64_t)b * s_max;

  // this lane's queries: column c16 of each of the wave's QG groups of 16
  int qk[QG], qpos[QG];
  bool qvalid[QG];
  bf16x8_t qf[QG][DS];
  f32x4_t o[QG][DB];
  float m_run[QG], l_run[QG];
#pragma unroll
  for (int qg = 0; qg < QG; ++qg) {
    const int qi = (wave * QG + qg) * 16 + c16;
    qvalid[qg] = qi < tile.y;
    qk[qg] = tile.x + (qvalid[qg] ? qi : 0);
    qpos[qg] = qvalid[qg] ? pos[rows[qk[qg]]] : -1;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const uint4 v =
          *reinterpret_cast<const uint4*>(q + (int64_t)qk[qg] * rs + h * HD + s * 32 + g * 8);
      qf[qg][s] = __builtin_bit_cast(bf16x8_t, v);
    }
#pragma unroll
    for (int i = 0; i < DB; ++i) o[qg][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m_run[qg] = -INFINITY;
    l_run[qg] = 0.0f;
  }

  const int nkb = pmax / KB + 1;
  for (int kb = 0; kb < nkb; ++kb) {
    const int t0 = kb * KB;
    // ---- stage K [64][HD] row-major; keys past pmax are zero
    constexpr int CH = HD / 8;  // 16-byte chunks per row
#pragma unroll
    for (int e = tid; e < KB * CH; e += 256) {
      const int r = e / CH, c = (e % CH) * 8;
      const int t = t0 + r;
      uint4 kv = make_uint4(0, 0, 0, 0);
      if (t <= pmax) kv = *reinterpret_cast<const uint4*>(kc + (kbase + t) * rs + h * HD + c);
      *reinterpret_cast<uint4*>(sK + r * KLD + c) = kv;
    }
    // ---- stage V^T [HD][64]: a thread takes 4 keys x 8 dims and writes eight
    // 8-byte runs (4 keys of one dim)
#pragma unroll
    for (int e = tid; e < (KB / 4) * CH; e += 256) {
      const int kg = e % (KB / 4), dc = e / (KB / 4);
      uint32_t w[4][4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int t = t0 + 4 * kg + kk;
        uint4 vv = make_uint4(0, 0, 0, 0);
        if (t <= pmax) vv = *reinterpret_cast<const uint4*>(vc + (kbase + t) * rs + h * HD + dc * 8);
        w[kk][0] = vv.x; w[kk][1] = vv.y; w[kk][2] = vv.z; w[kk][3] = vv.w;
      }
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        const int sh = (d & 1) * 16;
        const uint32_t e0 = (w[0][d >> 1] >> sh) & 0xffff, e1 = (w[1][d >> 1] >> sh) & 0xffff;
        const uint32_t e2 = (w[2][d >> 1] >> sh) & 0xffff, e3 = (w[3][d >> 1] >> sh) & 0xffff;
        *reinterpret_cast<uint2*>(sVt + (dc * 8 + d) * VLD + 4 * kg) =
            make_uint2(e0 | (e1 << 16), e2 | (e3 << 16));
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T: 4 key sub-blocks of 16; each K fragment serves QG groups
    f32x4_t s[QG][4];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
#pragma unroll
      for (int qg = 0; qg < QG; ++qg) s[qg][sb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const bf16x8_t a =
            *reinterpret_cast<const bf16x8_t*>(sK + (sb * 16 + c16) * KLD + ds * 32 + g * 8);
#pragma unroll
        for (int qg = 0; qg < QG; ++qg)
          s[qg][sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[qg][ds], s[qg][sb], 0, 0, 0);
      }
    }
    bf16x8_t pb[QG][2];
#pragma unroll
    for (int qg = 0; qg < QG; ++qg) {
      // ---- mask, running max
      float mloc = -INFINITY;
#pragma unroll
      for (int sb = 0; sb < 4; ++sb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int t = t0 + sb * 16 + g * 4 + v;
          float x = s[qg][sb][v] * scale_log2;
          x = (t <= qpos[qg]) ? x : -INFINITY;
          s[qg][sb][v] = x;
          mloc = fmaxf(mloc, x);
        }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
      const float m_new = fmaxf(m_run[qg], mloc);
      const float alpha = (m_new == -INFINITY) ? 1.0f : exp2f(m_run[qg] - m_new);
      m_run[qg] = m_new;
      l_run[qg] *= alpha;
#pragma unroll
      for (int i = 0; i < DB; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) o[qg][i][v] *= alpha;
      // ---- P = exp2(S - m) packed as the B operand (key order: sub-block pairs)
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        uint16_t pv[8];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float x = s[qg][2 * kp + hh][v];
            const float ev = (x == -INFINITY) ? 0.0f : exp2f(x - m_new);
            const bf16 eb = f2bf(ev);
            l_run[qg] += bf2f(eb);
            pv[hh * 4 + v] = eb;
          }
        pb[qg][kp] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(pv));
      }
    }
    // ---- O^T += V^T P^T; each V^T fragment serves QG groups
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        const bf16* vr = sVt + (db * 16 + c16) * VLD + kp * 32 + g * 4;
        const uint2 lo = *reinterpret_cast<const uint2*>(vr);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
        for (int qg = 0; qg < QG; ++qg)
          o[qg][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[qg][kp], o[qg][db], 0, 0, 0);
      }
    __syncthreads();
  }
#pragma unroll
  for (int qg = 0; qg < QG; ++qg) {
    float l = l_run[qg];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (!qvalid[qg]) continue;
    const float inv = 1.0f / l;
    bf16* dst = out + (int64_t)qk[qg] * rs + h * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int d0 = db * 16 + g * 4;
      const uint32_t w0 =
          (uint32_t)f2bf(o[qg][db][0] * inv) | ((uint32_t)f2bf(o[qg][db][1] * inv) << 16);
      const uint32_t w1 =
          (uint32_t)f2bf(o[qg][db][2] * inv) | ((uint32_t)f2bf(o[qg][db][3] * inv) << 16);
      *reinterpret_cast<uint2*>(dst + d0) = make_uint2(w0, w1);
    }
  }
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_attend_workspace_bytes(int max_active, int n_seq) {
  const size_t tiles = (size_t)(max_active / QT + n_seq + 1);
  return 256 + tiles * sizeof(int2);
}

extern "C" adept_status adept_attend(adept_dtype dt, int n_heads, int head_dim, float scale,
                                     int causal, const void* q, const int32_t* rows,
                                     const int32_t* n_active, int max_active, const int32_t* pos,
                                     const int32_t* seq, int n_seq, const void* k_layer,
                                     const void* v_layer, int s_max, const int32_t* key_len,
                                     const uint8_t* key_live, void* out, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "attend: bad dtype");
  ADEPT_REQUIRE(n_heads > 0 && head_dim > 0 && head_dim <= 128 && 256 % head_dim == 0,
                "attend: head_dim %d must divide 256 and be <= 128", head_dim);
  ADEPT_REQUIRE(max_active >= 0 && n_seq > 0 && s_max > 0, "attend: bad sizes");
  ADEPT_REQUIRE(s_max <= 16384, "attend: s_max %d above 16384", s_max);
  ADEPT_REQUIRE(q && rows && n_active && pos && seq && k_layer && v_layer && out,
                "attend: NULL tensor");
  ADEPT_REQUIRE(causal || key_len, "attend: bidirectional attention needs key_len");
  if (max_active == 0) return ADEPT_OK;
  hipStream_t s = as_stream(stream);
  const bool mfma = dt == ADEPT_BF16 && causal && !key_live && (head_dim == 64 || head_dim == 128);
  if (mfma && workspace) {
    const size_t need = adept_attend_workspace_bytes(max_active, n_seq);
    if (workspace_bytes < need) {
      set_error("attend: workspace of %zu bytes needed", need);
      return ADEPT_E_WORKSPACE;
    }
    ADEPT_REQUIRE(aligned16(q) && aligned16(k_layer) && aligned16(v_layer) && aligned16(out) &&
                      aligned16(workspace),
                  "attend: tensors must be 16-byte aligned");
    int32_t* n_tiles = (int32_t*)workspace;
    int2* tiles = (int2*)((char*)workspace + 256);
    const int max_tiles = max_active / QT + n_seq + 1;
    ADEPT_LAUNCH(attend_plan_kernel, dim3(1), dim3(1024), 2 * (n_seq + 1) * sizeof(int), s,
                       rows, n_active, max_active, seq, n_seq, tiles, n_tiles);
    ADEPT_CHECK_LAUNCH("attend_plan");
    const float sl = scale * 1.4426950408889634f;
    dim3 grid(max_tiles, n_heads);
    if (head_dim == 128)
      ADEPT_LAUNCH(attend_prefill_kernel<128>, grid, dim3(256), 0, s, n_heads, sl,
                         (const bf16*)q, rows, pos, seq, (const bf16*)k_layer,
                         (const bf16*)v_layer, s_max, tiles, n_tiles, (bf16*)out);
    else
      ADEPT_LAUNCH(attend_prefill_kernel<64>, grid, dim3(256), 0, s, n_heads, sl,
                         (const bf16*)q, rows, pos, seq, (const bf16*)k_layer,
                         (const bf16*)v_layer, s_max, tiles, n_tiles, (bf16*)out);
    return launch_status("attend_prefill");
  }
  const size_t smem = (size_t)(128 + s_max) * sizeof(float);
  dim3 grid(max_active, n_heads);
  if (dt == ADEPT_BF16)
    ADEPT_LAUNCH(attend_generic_kernel<bf16>, grid, dim3(kGenThreads), smem, s, n_heads,
                       head_dim, scale, causal, (const bf16*)q, rows, n_active, max_active, pos,
                       seq, (const bf16*)k_layer, (const bf16*)v_layer, s_max, key_len,
                       key_live, (bf16*)out);
  else
    ADEPT_LAUNCH(attend_generic_kernel<float>, grid, dim3(kGenThreads), smem, s, n_heads,
                       head_dim, scale, causal, (const float*)q, rows, n_active, max_active,
                       pos, seq, (const float*)k_layer, (const float*)v_layer, s_max, key_len,
                       key_live, (float*)out);
  return launch_status("attend_generic");
}
