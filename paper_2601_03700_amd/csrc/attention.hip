// Attention of the active tokens over one layer's cache, whose entries were
// either computed by the layer itself (tokens still active) or generated
// from an earlier exit state (Section 3, Eq. 5; Section 4.3).  The kernels do
// not distinguish the two: a generated entry is an ordinary cache row.
//
// Query tiles (bf16, head_dim 64/128; prefill, and the bidirectional
// attention of classification over the live keys): a plan kernel cuts the
// compacted query list into tiles of <= 128 consecutive entries of one
// sequence; a
// 256-thread workgroup takes one (tile, head), each wave two groups of 16
// queries, so every K/V fragment read from LDS feeds two MFMAs.  Key
// blocks of 64 rows are staged in LDS (K row-major, V transposed with packed
// 8-byte writes of 4 keys), and the
// scores are formed transposed, S^T = K Q^T, with v_mfma_f32_16x16x32_bf16 so
// that each lane owns one query column: the online softmax then needs only
// two cross-lane steps (lane swaps) for the running max, and the
// probabilities already sit in the B-operand layout of O^T += V^T P^T (the
// order of keys inside an MFMA's reduction is free, so V^T is read in the
// same key order).  The softmax is the VALU side of the loop, so it is kept
// short: v_max3 without input quieting, the normaliser as bf16 dot products,
// and a reference max that moves (and O is rescaled) only when a block's
// max exceeds it by more than 2^8.
//
// Key chunks (bf16, few queries per sequence: decode): see
// attend_split_kernel.  Generic path (f32): one workgroup per (query, head),
// scores for all keys in LDS, exact softmax, then a weighted sum of V rows.
#include <algorithm>

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
// prefill plan: tiles of <= QT consecutive query entries of one sequence
// ---------------------------------------------------------------------------
constexpr int QT = 128;  // queries per tile (4 waves x 2 groups of 16)
constexpr int kPrefillThreads = 256;
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
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
constexpr bf16x2_t kOnes2 = {(__bf16)1.0f, (__bf16)1.0f};
constexpr float kLazy = 8.0f;   // log2 headroom of the reference max

// max(a, b, c) in one v_max3_f32.  The scores come from MFMAs, which the
// compiler cannot prove canonical, so fmaxf would first quiet each input
// (one extra v_max per value); finite values and -inf need no quieting.
__device__ __forceinline__ float max3_raw(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Max over the four lanes l, l^16, l^32, l^48 that hold one column of a
// 16x16 MFMA result: each lane swap gives every lane its partner row's value
// in one of its two results.
__device__ __forceinline__ float max_column(float m) {
  uint32_t u = __float_as_uint(m);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  m = max3_raw(m, __uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(m);
  const auto b = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return max3_raw(m, __uint_as_float(b[0]), __uint_as_float(b[1]));
}
// causal: keys 0..pos of each query; else keys 0..key_len[b]-1 of the
// sequence, all of them for every query (bidirectional).  key_live
// (nullable) drops keys whose byte is 0.
//
// One workgroup per (tile of <= 128 queries of one sequence, head); each of
// the four waves holds two groups of 16 queries, so every K and V fragment
// read from LDS serves two MFMAs, and two workgroups share a CU, so one
// wave's softmax overlaps the other's MFMAs on each SIMD.  K and V advance
// in blocks of 64 keys through two LDS stages filled by direct
// global->LDS loads: the loads of block kb+1 are issued before block kb is
// computed, and one barrier per block publishes the next stage and retires
// the current one.  V stays row-major in LDS; the A operand of O^T = V^T P^T
// is read with the LDS transpose read.
template <int HD>
__global__ __launch_bounds__(kPrefillThreads, 2) void attend_prefill_kernel(
    int H, float scale_log2, int causal, const bf16* __restrict__ q,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ pos,
    const int32_t* __restrict__ seq, const bf16* __restrict__ kc, const bf16* __restrict__ vc,
    int s_max, const int32_t* __restrict__ key_len, const uint8_t* __restrict__ key_live,
    const int2* __restrict__ tiles, const int32_t* __restrict__ n_tiles, int max_tiles,
    bf16* __restrict__ out) {
  constexpr int NT = kPrefillThreads;
  constexpr int DS = HD / 32;               // 32-wide dim steps for S
  constexpr int DB = HD / 16;               // 16-row dim blocks of O^T
  constexpr int QG = QT / (16 * (NT / 64)); // 16-query groups per wave
  constexpr int ROWB = HD * 2;              // bytes per K or V row
  constexpr int NCH = ROWB / 16;            // 16-byte chunks per row
  constexpr int RPI = 1024 / ROWB;          // rows per direct-load instruction
  constexpr int BLK = KB * ROWB;            // bytes of one block of K (or V)
  constexpr int DPW = (KB / RPI) / (NT / 64);   // direct loads per wave and operand
  static_assert(DPW >= 1 && (KB / RPI) % (NT / 64) == 0, "block splits over the waves");
  // [stage][K = 0, V = 1][block]
  __shared__ __attribute__((aligned(1024))) char sKV[2][2][BLK];
  __shared__ uint64_t sLive[2];

  // Work item of this workgroup.  The hardware deals consecutive workgroup
  // ids round-robin to the 8 XCDs; with several heads (1-D grid, heads
  // padded to a multiple of 8), XCD x takes heads x, x+8, ... one after
  // another, each head's tiles longest first, so the tiles in flight on an
  // XCD share a few sequences' K/V in its L2.  One head: blockIdx.x = tile.
  const int nt = *n_tiles;
  int ti, h;
  if (gridDim.y == 1 && H > 1) {
    const int k = blockIdx.x >> 3;
    ti = k % max_tiles;
    h = (blockIdx.x & 7) + 8 * (k / max_tiles);
    if (h >= H) return;
  } else {
    ti = blockIdx.x;
    h = blockIdx.y;
  }
  if (ti >= nt) return;
  const int2 tile = tiles[nt - 1 - ti];   // longest (latest) tiles first
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int64_t rs = (int64_t)H * HD;

  const int b = seq[rows[tile.x]];
  // keys [0, tend) are read; causal queries mask t > pos themselves
  const int tend = causal ? pos[rows[tile.x + tile.y - 1]] + 1 : min(key_len[b], s_max);
  const int64_t kbase = (int64_t)b * s_max;

  // this lane's queries: column c16 of each of the wave's QG groups of 16
  int qk[QG], qpos[QG];
  bool qvalid[QG];
  bf16x8_t qf[QG][DS];
  f32x4_t o[QG][DB];
  float m_ref[QG], l_run[QG];
#pragma unroll
  for (int qg = 0; qg < QG; ++qg) {
    const int qi = (wave * QG + qg) * 16 + c16;
    qvalid[qg] = qi < tile.y;
    qk[qg] = tile.x + (qvalid[qg] ? qi : 0);
    qpos[qg] = qvalid[qg] ? (causal ? pos[rows[qk[qg]]] : tend - 1) : -1;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const uint4 v =
          *reinterpret_cast<const uint4*>(q + (int64_t)qk[qg] * rs + h * HD + s * 32 + g * 8);
      qf[qg][s] = __builtin_bit_cast(bf16x8_t, v);
    }
#pragma unroll
    for (int i = 0; i < DB; ++i) o[qg][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m_ref[qg] = -INFINITY;
    l_run[qg] = 0.0f;
  }
  // smallest position among the wave's valid queries: blocks of keys at or
  // below it (and inside the range, without a live-key mask) need no mask
  int wmin = INT_MAX;
#pragma unroll
  for (int qg = 0; qg < QG; ++qg) wmin = min(wmin, qvalid[qg] ? qpos[qg] : INT_MAX);
  wmin = min(wmin, __shfl_xor(wmin, 1, 64));
  wmin = min(wmin, __shfl_xor(wmin, 2, 64));
  wmin = min(wmin, __shfl_xor(wmin, 4, 64));
  wmin = min(wmin, __shfl_xor(wmin, 8, 64));

  // ---- K and V blocks reach LDS by direct global->LDS loads (lane l of an
  // instruction writes 16 bytes at base + 16 l, i.e. RPI whole rows), two
  // stages deep.  The 16-byte chunk c of row r is stored at position
  // c ^ fK(r) (K) or c ^ fV(r) (V): the K fragment reads (16 rows, one
  // chunk) and the V transpose reads (4 rows x 2 chunks per 16 lanes) then
  // fall on distinct banks.  Keys past the range re-read the range's last
  // key: finite values the mask gives weight 0.
  auto fK = [](int r) { return HD == 128 ? (r & 15) : ((r >> 1) & 7); };
  auto fV = [](int r) { return HD == 128 ? 2 * (r & 7) : 2 * ((r >> 1) & 3); };
  // Byte offsets of this lane's loads from a block's first key row: the row
  // part (same for K and V) and the chunk part.  A block's base address is
  // uniform, so each load is one scalar base plus one 32-bit lane offset.
  const uint32_t rowb = (uint32_t)(rs * 2);
  uint32_t lrow[DPW], lcol[2][DPW];
#pragma unroll
  for (int j = 0; j < DPW; ++j) {
    const int r = (wave * DPW + j) * RPI + lane / NCH;
    lrow[j] = (uint32_t)r * rowb;
    lcol[0][j] = (uint32_t)(((lane % NCH) ^ fK(r)) * 16);
    lcol[1][j] = (uint32_t)(((lane % NCH) ^ fV(r)) * 16);
  }
  auto issue = [&](int kb, int u) {
    const int t0 = kb * KB;
    // rows past the range re-read its last row (the last block only)
    const uint32_t lim = t0 + KB > tend ? (uint32_t)(tend - 1 - t0) * rowb : 0xffffffffu;
#pragma unroll
    for (int op = 0; op < 2; ++op) {
      const char* blk = reinterpret_cast<const char*>((op ? vc : kc) + (kbase + t0) * rs + h * HD);
#pragma unroll
      for (int j = 0; j < DPW; ++j) {
        const int qd = wave * DPW + j;
        const uint32_t off = min(lrow[j], lim) + lcol[op][j];
        __builtin_amdgcn_global_load_lds(
            (__attribute__((address_space(1))) void*)(blk + off),
            (__attribute__((address_space(3))) void*)(&sKV[u][op][qd * 1024]), 16, 0, 0);
      }
    }
    if (key_live && wave == 0) {
      const bool lv = t0 + lane < tend && key_live[kbase + min(t0 + lane, tend - 1)] != 0;
      const uint64_t m = __ballot(lv);
      if (lane == 0) sLive[u] = m;
    }
  };
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

  const int nkb = (tend + KB - 1) / KB;
  if (nkb > 0) issue(0, 0);
  __syncthreads();   // waits for every wave's loads, then publishes stage 0
  for (int kb = 0; kb < nkb; ++kb) {
    const int u = kb & 1;
    const int t0 = kb * KB;
    // the other stage was last read in block kb-1, which every wave
    // finished before the previous barrier
    if (kb + 1 < nkb) issue(kb + 1, u ^ 1);
    const char* cK = sKV[u][0];
    const char* cV = sKV[u][1];

    // ---- S^T = K Q^T: 4 key sub-blocks of 16; each K fragment serves QG groups.
    // The matrix phases run at a raised wave priority, so the SIMD's other
    // wave (in its softmax) takes the issue slots the MFMAs leave free.
    __builtin_amdgcn_s_setprio(1);
    f32x4_t s[QG][4];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
#pragma unroll
      for (int qg = 0; qg < QG; ++qg) s[qg][sb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const int r = sb * 16 + c16;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
            cK + r * ROWB + ((4 * ds + g) ^ fK(r)) * 16);
#pragma unroll
        for (int qg = 0; qg < QG; ++qg)
          s[qg][sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[qg][ds], s[qg][sb], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    // ---- mask (only blocks that reach past a query's position, past the
    // range, or under a live-key mask), in the exp2 domain
    const bool full = !key_live && t0 + KB <= tend && t0 + KB - 1 <= wmin;
    if (!full) {
      const uint64_t lm = key_live ? sLive[u] : ~0ull;
#pragma unroll
      for (int qg = 0; qg < QG; ++qg)
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int kl = sb * 16 + g * 4 + v;
            const bool keep = t0 + kl <= qpos[qg] && ((lm >> kl) & 1);
            s[qg][sb][v] = keep ? s[qg][sb][v] : -INFINITY;
          }
    }
    // ---- running max of the block per query column: each lane folds its 16
    // scores of a group with v_max3, then the four lanes of the column
    // (l, l^16, l^32, l^48) by two lane swaps (the max of the raw scores is
    // taken first and scaled once: scale > 0)
    float mblk[QG];
    bool need = false;
#pragma unroll
    for (int qg = 0; qg < QG; ++qg) {
      float m = max3_raw(s[qg][0][0], s[qg][0][1], s[qg][0][2]);
      m = max3_raw(m, s[qg][0][3], s[qg][1][0]);
      m = max3_raw(m, s[qg][1][1], s[qg][1][2]);
      m = max3_raw(m, s[qg][1][3], s[qg][2][0]);
      m = max3_raw(m, s[qg][2][1], s[qg][2][2]);
      m = max3_raw(m, s[qg][2][3], s[qg][3][0]);
      m = max3_raw(m, s[qg][3][1], s[qg][3][2]);
      m = max_column(max3_raw(m, s[qg][3][3], m)) * scale_log2;
      mblk[qg] = m;
      // the reference max moves only when the block exceeds it by more than
      // 2^kLazy: the weights exp2(s - m_ref) then stay below 2^kLazy, and
      // the result (O / l, both taken against the same reference) is the same
      need |= m > m_ref[qg] + kLazy;
    }
    if (__any(need)) {
#pragma unroll
      for (int qg = 0; qg < QG; ++qg) {
        const float m_new = fmaxf(m_ref[qg], mblk[qg]);
        const float alpha = m_new == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f(m_ref[qg] - m_new);
        m_ref[qg] = m_new;
        l_run[qg] *= alpha;
#pragma unroll
        for (int i = 0; i < DB; ++i)
#pragma unroll
          for (int v = 0; v < 4; ++v) o[qg][i][v] *= alpha;
      }
    }
    // ---- P = exp2(S * scale - m_ref) packed as the B operand (key order:
    // sub-block pairs); a masked score (-inf) gives exp2(-inf) = 0.  The
    // normaliser sums the rounded weights the MFMA multiplies (a bf16 dot
    // product of each packed pair with (1, 1)).
    bf16x8_t pb[QG][2];
#pragma unroll
    for (int qg = 0; qg < QG; ++qg) {
      const float msub = m_ref[qg] == -INFINITY ? 0.0f : m_ref[qg];
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        uint32_t pw[4];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int v = 0; v < 4; v += 2) {
            const float e0 =
                __builtin_amdgcn_exp2f(fmaf(s[qg][2 * kp + hh][v], scale_log2, -msub));
            const float e1 =
                __builtin_amdgcn_exp2f(fmaf(s[qg][2 * kp + hh][v + 1], scale_log2, -msub));
            const uint32_t w = pack_bf16x2(e0, e1);
            l_run[qg] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w), kOnes2,
                                                        l_run[qg], false);
            pw[hh * 2 + v / 2] = w;
          }
        pb[qg][kp] = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
      }
    }
    __builtin_amdgcn_s_setprio(1);
    // ---- O^T += V^T P^T; each V^T fragment serves QG groups.  The A operand
    // (16 dims x 32 keys) comes from row-major V by two transpose reads: in
    // each 16-lane group, source lane L reads 4 dims of key k0 + L/4 and
    // lane i receives dim n0 + i of keys k0..k0+3, k0 = 32 kp + 16 hh + 4 g,
    // which is the key order of P.
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        s16x4 half[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int r = 32 * kp + 16 * hh + 4 * g + (c16 >> 2);
          const int c = 2 * db + ((c16 & 3) >> 1);
          const char* pa = cV + r * ROWB + ((c ^ fV(r)) * 16) + 8 * (c16 & 1);
          half[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)pa);
        }
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, __builtin_shufflevector(half[0], half[1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int qg = 0; qg < QG; ++qg)
          o[qg][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[qg][kp], o[qg][db], 0, 0, 0);
      }
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();   // stage kb+1 landed (every wave waited for its loads); stage u retired
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


// ---------------------------------------------------------------------------
// split-K kernel (decode and bidirectional): HBM-bound streaming of K/V rows
// ---------------------------------------------------------------------------
constexpr int kSplitThreads = 256;

// Workgroups of a decode attention launch: about 8192 for 128-wide heads and
// 2048 for 64-wide ones (a workgroup then takes twice the keys per pass of
// its lane groups; measured best for each width).
__host__ __device__ inline int64_t split_target(int hd) { return hd <= 64 ? 2048 : 8192; }

// Chunks per (query entry, head) for n entries: about split_target(hd)
// workgroups, at most one chunk per 256 keys of s_max.  The host sizes the
// grid and the workspace for max_active entries (nc_host chunks); the
// kernels take the chunk count from the device count n <= max_active, which
// gives more chunks when fewer entries are active (a fuller grid), within the
// grid and workspace capacity max_active * nc_host.  nc_host == 1 (the output
// is written directly, no combine) stays 1.
__host__ __device__ inline int split_nc(int n, int H, int hd, int s_max) {
  const int64_t pairs = (int64_t)(n > 1 ? n : 1) * H;
  const int64_t want = (split_target(hd) + pairs - 1) / pairs;
  const int64_t most = (s_max + 255) / 256;
  return (int)(want < 1 ? 1 : (want < most ? want : (most < 1 ? 1 : most)));
}
__device__ inline int split_nc_dev(int n, int max_active, int nc_host, int H, int hd, int s_max) {
  if (nc_host == 1 || n <= 0) return nc_host;
  const int cap = (int)(((int64_t)max_active * nc_host) / n);
  const int f = split_nc(n, H, hd, s_max);
  return max(nc_host, min(f, cap));
}

// Workgroup (k, c, h): keys [c*CK, min(L, (c+1)*CK)) of query entry k, head
// h, CK = ceil(L / nc), nc = split_nc_dev of the device count (nc_host: the
// count the grid was sized with).  A key's row of head h (HD bf16 = HD*2 bytes) is read
// by LPK = HD/8 lanes, 16 bytes each (non-temporal: nothing reads it again
// while cached), so every load instruction covers whole rows; the wave's GPW lane groups take different keys, four per group in
// flight.  Scores are q.k over the group (xor shuffles), and each group keeps
// an online softmax in the exp2 domain (q is pre-scaled by scale*log2(e)).
// The workgroup's groups are merged in LDS; with one chunk the output is
// written directly, else (max, sum, unnormalised o) go to the workspace for
// attend_combine_kernel.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int HD>
__global__ __launch_bounds__(kSplitThreads) void attend_split_kernel(
    int H, float scale_log2, int causal, int nc_host, const bf16* __restrict__ q,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ n_active, int max_active,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ seq,
    const bf16* __restrict__ kc, const bf16* __restrict__ vc, int s_max,
    const int32_t* __restrict__ key_len, const uint8_t* __restrict__ key_live,
    bf16* __restrict__ out, float* __restrict__ part) {
  constexpr int LPK = HD / 8;                 // lanes per key row
  constexpr int GPW = 64 / LPK;               // key groups per wave
  constexpr int G = GPW * (kSplitThreads / 64);
  __shared__ float gm[G], gl[G];
  __shared__ float go[G][HD + 4];
  const int na = min(*n_active, max_active);
  const int nc = split_nc_dev(na, max_active, nc_host, H, HD, s_max);
  const int k = blockIdx.x / nc, c = blockIdx.x - (blockIdx.x / nc) * nc, h = blockIdx.y;
  if (k >= na) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int grp = (tid >> 6) * GPW + lane / LPK;   // key group in the workgroup
  const int sub = lane % LPK;                      // 8-dim slice of the row
  const int row = rows[k];
  const int b = seq[row];
  const int L = min(causal ? pos[row] + 1 : key_len[b], s_max);
  const int ck = (L + nc - 1) / nc;
  const int t0 = c * ck, t1 = min(L, t0 + ck);
  const int64_t rs = (int64_t)H * HD;               // cache row stride (elements)
  const bf16* kb = kc + (int64_t)b * s_max * rs + h * HD + sub * 8;
  const bf16* vb = vc + (int64_t)b * s_max * rs + h * HD + sub * 8;
  const uint8_t* live = key_live ? key_live + (int64_t)b * s_max : nullptr;

  float qf[8];
  {
    const uint4 qv = *reinterpret_cast<const uint4*>(q + (int64_t)k * rs + h * HD + sub * 8);
    const uint32_t w[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      qf[2 * e] = __uint_as_float(w[e] << 16) * scale_log2;
      qf[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u) * scale_log2;
    }
  }
  float m = -INFINITY, l = 0.0f, o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = 0.0f;
  for (int tb = t0 + grp; tb < t1; tb += 4 * G) {
    uint4 kv[4], vv[4];
    bool ok[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = tb + u * G;
      ok[u] = t < t1;
      const int tt = ok[u] ? t : t0;            // clamped: loaded, never used
      // streaming: a key row is read once per (query, head)
      const u32x4_t kn = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(kb + (int64_t)tt * rs));
      const u32x4_t vn = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(vb + (int64_t)tt * rs));
      kv[u] = make_uint4(kn.x, kn.y, kn.z, kn.w);
      vv[u] = make_uint4(vn.x, vn.y, vn.z, vn.w);
    }
    float sc[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t w[4] = {kv[u].x, kv[u].y, kv[u].z, kv[u].w};
      float d = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        d = fmaf(qf[2 * e], __uint_as_float(w[e] << 16), d);
        d = fmaf(qf[2 * e + 1], __uint_as_float(w[e] & 0xffff0000u), d);
      }
#pragma unroll
      for (int off = LPK / 2; off > 0; off >>= 1) d += __shfl_xor(d, off, 64);
      const int t = tb + u * G;
      const bool use = ok[u] && (!live || live[ok[u] ? t : t0]);
      sc[u] = use ? d : -INFINITY;
    }
    const float mb = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    const float mn = fmaxf(m, mb);
    if (mn == -INFINITY) continue;              // nothing live yet in this group
    const float cf = exp2f(m - mn);             // m = -inf -> 0
    l *= cf;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] *= cf;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float pu = exp2f(sc[u] - mn);       // masked -> 0
      l += pu;
      const uint32_t w[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[2 * e] = fmaf(pu, __uint_as_float(w[e] << 16), o[2 * e]);
        o[2 * e + 1] = fmaf(pu, __uint_as_float(w[e] & 0xffff0000u), o[2 * e + 1]);
      }
    }
    m = mn;
  }
  // merge the workgroup's G groups
  if (sub == 0) {
    gm[grp] = m;
    gl[grp] = l;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) go[grp][sub * 8 + e] = o[e];
  __syncthreads();
  if (tid < HD) {
    float M = -INFINITY;
    for (int g = 0; g < G; ++g) M = fmaxf(M, gm[g]);
    float Ls = 0.0f, O = 0.0f;
    if (M != -INFINITY) {
      for (int g = 0; g < G; ++g) {
        const float w = exp2f(gm[g] - M);       // empty group: -inf -> 0
        Ls = fmaf(w, gl[g], Ls);
        O = fmaf(w, go[g][tid], O);
      }
    }
    const int64_t pq = (int64_t)k * H + h;
    if (nc == 1) {
      out[pq * HD + tid] = f2bf(O / Ls);
    } else {
      float* pp = part + (pq * nc + c) * (HD + 2);
      pp[2 + tid] = O;
      if (tid == 0) {
        pp[0] = M;
        pp[1] = Ls;
      }
    }
  }
}

// Merges the nc partial results of each (query entry, head).
template <int HD>
__global__ __launch_bounds__(HD) void attend_combine_kernel(int H, int nc_host,
                                                           const int32_t* __restrict__ n_active,
                                                           int max_active, int s_max,
                                                           const float* __restrict__ part,
                                                           bf16* __restrict__ out) {
  const int k = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
  const int na = min(*n_active, max_active);
  if (k >= na) return;
  const int nc = split_nc_dev(na, max_active, nc_host, H, HD, s_max);
  const int64_t pq = (int64_t)k * H + h;
  const float* pp = part + pq * nc * (HD + 2);
  // the chunks' loads are independent: unrolled so that they are in flight together
  float M = -INFINITY;
#pragma unroll 8
  for (int c = 0; c < nc; ++c) M = fmaxf(M, pp[c * (HD + 2)]);
  float Ls = 0.0f, O = 0.0f;
  if (M != -INFINITY) {
#pragma unroll 8
    for (int c = 0; c < nc; ++c) {
      const float* pc = pp + c * (HD + 2);
      const float w = exp2f(pc[0] - M);
      Ls = fmaf(w, pc[1], Ls);
      O = fmaf(w, pc[2 + d], O);
    }
  }
  out[pq * HD + d] = f2bf(O / Ls);
}

// Chunks per (query entry, head) the split kernel's grid is sized with.
int split_chunks(int max_active, int H, int hd, int s_max) {
  return split_nc(max_active, H, hd, s_max);
}

size_t split_workspace_bytes(int max_active, int H, int hd, int s_max) {
  const int nc = split_chunks(max_active, H, hd, s_max);
  return nc == 1 ? 0 : (size_t)max_active * H * nc * (hd + 2) * sizeof(float);
}

}  // namespace
}  // namespace adept

using namespace adept;

namespace adept {

size_t attend_workspace_bytes(int max_active, int n_seq, int n_heads, int head_dim, int s_max) {
  const size_t tiles = 256 + (size_t)(max_active / QT + n_seq + 1) * sizeof(int2);
  return std::max(tiles, split_workspace_bytes(max_active, n_heads, head_dim, s_max));
}

adept_status attend_dispatch(adept_dtype dt, int n_heads, int head_dim, float scale, int causal,
                             const void* q, const int32_t* rows, const int32_t* n_active,
                             int max_active, const int32_t* pos, const int32_t* seq, int n_seq,
                             const void* k_layer, const void* v_layer, int s_max,
                             const int32_t* key_len, const uint8_t* key_live, void* out,
                             void* workspace, size_t workspace_bytes, bool allow_tiles,
                             hipStream_t s) {
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "attend: bad dtype");
  ADEPT_REQUIRE(n_heads > 0 && head_dim > 0 && head_dim <= 128 && 256 % head_dim == 0,
                "attend: head_dim %d must divide 256 and be <= 128", head_dim);
  ADEPT_REQUIRE(max_active >= 0 && n_seq > 0 && s_max > 0, "attend: bad sizes");
  ADEPT_REQUIRE(s_max <= 16384, "attend: s_max %d above 16384", s_max);
  ADEPT_REQUIRE(q && rows && n_active && pos && seq && k_layer && v_layer && out,
                "attend: NULL tensor");
  ADEPT_REQUIRE(causal || key_len, "attend: bidirectional attention needs key_len");
  if (max_active == 0) return ADEPT_OK;
  const bool fast = dt == ADEPT_BF16 && (head_dim == 64 || head_dim == 128) && workspace;
  if (fast) {
    const size_t need = attend_workspace_bytes(max_active, n_seq, n_heads, head_dim, s_max);
    if (workspace_bytes < need) {
      set_error("attend: workspace of %zu bytes needed", need);
      return ADEPT_E_WORKSPACE;
    }
    ADEPT_REQUIRE(aligned16(q) && aligned16(k_layer) && aligned16(v_layer) && aligned16(out) &&
                      aligned16(workspace),
                  "attend: tensors must be 16-byte aligned");
  }
  const float sl = scale * 1.4426950408889634f;   // scores in the exp2 domain
  // query tiles pay off when the queries of a sequence are many (prefill)
  if (fast && allow_tiles && max_active >= 4 * n_seq) {
    int32_t* n_tiles = (int32_t*)workspace;
    int2* tiles = (int2*)((char*)workspace + 256);
    const int max_tiles = max_active / QT + n_seq + 1;
    ADEPT_LAUNCH(attend_plan_kernel, dim3(1), dim3(1024), 2 * (n_seq + 1) * sizeof(int), s,
                 rows, n_active, max_active, seq, n_seq, tiles, n_tiles);
    ADEPT_CHECK_LAUNCH("attend_plan");
    // more than one head: 1-D grid in XCD-major order, the heads padded to a
    // multiple of 8 (the padding's workgroups return at once)
    const int h8 = (n_heads + 7) / 8 * 8;
    const dim3 grid = n_heads > 1 ? dim3(max_tiles * h8) : dim3(max_tiles, 1);
    if (head_dim == 128)
      ADEPT_LAUNCH(attend_prefill_kernel<128>, grid, dim3(kPrefillThreads), 0, s, n_heads, sl, causal,
                   (const bf16*)q, rows, pos, seq, (const bf16*)k_layer, (const bf16*)v_layer,
                   s_max, key_len, key_live, tiles, n_tiles, max_tiles, (bf16*)out);
    else
      ADEPT_LAUNCH(attend_prefill_kernel<64>, grid, dim3(kPrefillThreads), 0, s, n_heads, sl, causal,
                   (const bf16*)q, rows, pos, seq, (const bf16*)k_layer, (const bf16*)v_layer,
                   s_max, key_len, key_live, tiles, n_tiles, max_tiles, (bf16*)out);
    return launch_status("attend_prefill");
  }
  if (fast) {
    const int nc = split_chunks(max_active, n_heads, head_dim, s_max);
    float* part = (float*)workspace;
    dim3 grid(max_active * nc, n_heads);
    if (head_dim == 128)
      ADEPT_LAUNCH(attend_split_kernel<128>, grid, dim3(kSplitThreads), 0, s, n_heads, sl,
                   causal, nc, (const bf16*)q, rows, n_active, max_active, pos, seq,
                   (const bf16*)k_layer, (const bf16*)v_layer, s_max, key_len, key_live,
                   (bf16*)out, part);
    else
      ADEPT_LAUNCH(attend_split_kernel<64>, grid, dim3(kSplitThreads), 0, s, n_heads, sl,
                   causal, nc, (const bf16*)q, rows, n_active, max_active, pos, seq,
                   (const bf16*)k_layer, (const bf16*)v_layer, s_max, key_len, key_live,
                   (bf16*)out, part);
    ADEPT_CHECK_LAUNCH("attend_split");
    if (nc > 1) {
      dim3 g2(max_active, n_heads);
      if (head_dim == 128)
        ADEPT_LAUNCH(attend_combine_kernel<128>, g2, dim3(128), 0, s, n_heads, nc, n_active,
                     max_active, s_max, part, (bf16*)out);
      else
        ADEPT_LAUNCH(attend_combine_kernel<64>, g2, dim3(64), 0, s, n_heads, nc, n_active,
                     max_active, s_max, part, (bf16*)out);
    }
    return launch_status("attend_split");
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

}  // namespace adept

extern "C" size_t adept_attend_workspace_bytes(int max_active, int n_seq, int n_heads,
                                               int head_dim, int s_max) {
  return attend_workspace_bytes(max_active, n_seq, n_heads, head_dim, s_max);
}

extern "C" adept_status adept_attend(adept_dtype dt, int n_heads, int head_dim, float scale,
                                     int causal, const void* q, const int32_t* rows,
                                     const int32_t* n_active, int max_active, const int32_t* pos,
                                     const int32_t* seq, int n_seq, const void* k_layer,
                                     const void* v_layer, int s_max, const int32_t* key_len,
                                     const uint8_t* key_live, void* out, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  return attend_dispatch(dt, n_heads, head_dim, scale, causal, q, rows, n_active, max_active,
                         pos, seq, n_seq, k_layer, v_layer, s_max, key_len, key_live, out,
                         workspace, workspace_bytes, true, as_stream(stream));
}
