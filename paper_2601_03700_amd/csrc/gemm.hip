// Dense and grouped GEMMs of the hot path, C[m][n] = sum_k A[m][k] B[n][k]
// (B in nn.Linear [out][in] order, so both operands are K-contiguous).
//
// bf16 path: one 256-thread workgroup computes a 256x256 output tile with
// v_mfma_f32_32x32x16_bf16; its four waves each own a 128x128 sub-tile
// (4x4 MFMA blocks, 256 accumulators per lane, held in AGPRs).  K advances
// 64 at a time.  Operands reach LDS by direct global->LDS loads
// (global_load_lds_dwordx4: lane l of an instruction lands 16 bytes at base
// + 16 l), eight lanes per 128-byte row, so every row of a stage is one whole
// cache line: the load path sustains about 1.5x the bytes per cycle it does
// with half-line requests.  The LDS (160 KiB) is a ring of five 32 KiB slots,
// one operand of one stage each; while stage k is consumed, B of stage k+1
// and A of stage k+2 are in flight, so the loads that miss L2 have one to
// two stages of MFMA work (2048 cycles each) to land.  Within a row the
// eight 16-byte chunks are permuted, chunk c of row r at position
// c ^ ((r >> 1) & 7): LDS serves a 16-byte read for 16 lanes per cycle
// (64 banks), the 16 rows of such a read fall into the two bank halves by
// r mod 2, and the permutation gives the 8 rows of a half 8 distinct chunk
// positions, so the operand reads are free of bank conflicts.  The operand
// fragments of the next k step are read while the current step's MFMAs run,
// and the loads of later stages are issued between MFMAs; one vmcnt wait and
// one barrier per stage order the ring.
//
// Workgroups are mapped to tiles XCD by XCD: the hardware deals consecutive
// workgroup ids round-robin to the 8 XCDs, so the id is remapped to give each
// XCD a contiguous block of tiles, rastered in groups of 8 row tiles; the
// workgroups resident on one XCD then share A and B k-slices in its L2.
//
// Row gathers (active-row lists) are folded into the per-lane load
// addresses.  The epilogue stages the accumulators through LDS, 32 rows of a
// wave at a time, so that its global loads and stores cover whole rows; a
// per-row scale (1/rms of the row, with the norm gain folded into B
// beforehand) is applied first, then RoPE + cache store (the wave's 128
// columns cover whole heads of 64 or 128, so a column's rotary partner is in
// the same staged row), residual add, SwiGLU (B tile = 64 gate rows + 64 up
// rows per wave), or plain store.
//
// The grouped variant is the decoupled KV generation of Eq. 9: one
// workgroup per (layer r, 256-row tile, column tile) item, the items built on
// the device from the exited rows sorted by exit layer (rows with i* < r form
// a prefix); B is [Wk_r; Wv_r] with layer r's gain folded in, the row scale is
// 1/rms(s~), and the epilogue writes K (with RoPE) and V into cache[r].
//
// f32 path (small configurations only): a plain 64x64-tiled FMA GEMM into a
// float scratch buffer followed by an element-wise epilogue kernel.
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace adept {
namespace {

constexpr int BM = 256, BN = 256;
constexpr int BK = 64;                                          // k columns per stage: 128-byte rows
constexpr int kSlots = 5;                                       // LDS ring slots, one operand each
constexpr int kThreads = 256;
constexpr int kStageBytes = BM * BK * 2;                        // one operand, one stage: 32 KiB
constexpr size_t kLdsBytes = (size_t)kSlots * kStageBytes;     // 160 KiB: all of a CU's LDS
constexpr int kEpiStride = 136;                                 // floats per staged epilogue row
constexpr int kEpiWaveBytes = 32 * kEpiStride * 4;              // one wave's 32 staged rows
constexpr int kEpiMetaBytes = 128 * 3 * 4;                      // per-row scale, row/slot, position
static_assert(4 * (kEpiWaveBytes + kEpiMetaBytes) <= (int)kLdsBytes,
              "epilogue staging fits in the ring");

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) char lds_char_t;
typedef __attribute__((address_space(3))) const bf16x8_t lds_bf16x8_t;
typedef __attribute__((address_space(1))) void glb_void_t;

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
  const float* row_scale;   // [compact m] or nullptr
  const int32_t* rows;
  const bf16* resid;
  const bf16* bias;         // [N] or nullptr
  const int32_t* pos;
  const int32_t* slot;
  const float* rope_cos;
  const float* rope_sin;
  int head_dim, d_q;
  bf16* q_out;
  bf16* k_cache;
  bf16* v_cache;
  int tiles_m, tiles_n;
  // grouped (KV generation)
  const int32_t* work;      // packed (layer << 16) | m_tile
  const int32_t* n_work;
  const int32_t* grp_m;     // [N+2]: rows with exit layer < r
  const int32_t* srows;     // exited rows sorted by exit layer
  int64_t b_layer_stride;
  int64_t cache_layer_stride;
  int64_t bias_layer_stride; // grouped: layer r's bias at bias + (r-1) * stride
  int a_sorted;             // grouped: A holds the rows in sorted order (row m), not by token
  // per-row second A buffer: token row r reads A2 when a_sel[r] & 1 (nullable)
  const bf16* A2;
  const int32_t* a_sel;
  float* rinv_out;          // skinny RESID: 1/rms of each result row (nullable)
  bf16* ln_out;             // skinny RESID: LayerNorm of each result row (nullable)
  float row_eps;
  RowExit ex;               // skinny RESID: the exit test of each result row (has_exit)
  int has_exit;
};

// x * sigmoid(x) with the hardware reciprocal (about 1 ulp in f32, far below
// the bf16 rounding of the output)
__device__ __forceinline__ float silu(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

// x * Phi(x) with the exact erf form of the normal CDF
__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.7071067811865476f));
}

// x * Phi(x) with the tanh approximation of the normal CDF (GPT-2's MLP)
__device__ __forceinline__ float gelu_tanh(float x) {
  return 0.5f * x * (1.0f + tanhf(0.7978845608028654f * fmaf(0.044715f * x, x * x, x)));
}

// Four bias values of columns c..c+3 (zeros when there is no bias).
__device__ __forceinline__ float4 bias4(const bf16* b, int64_t c) {
  if (!b) return make_float4(0.f, 0.f, 0.f, 0.f);
  const bf16x4_t v = *reinterpret_cast<const bf16x4_t*>(b + c);
  return make_float4(bf2f(v[0]), bf2f(v[1]), bf2f(v[2]), bf2f(v[3]));
}

__device__ __forceinline__ void dma16(const bf16* g, char* l) {
  __builtin_amdgcn_global_load_lds((glb_void_t*)g, (lds_void_t*)l, 16, 0, 0);
}

// s_waitcnt immediate (gfx9 encoding) that waits for all LDS operations and
// leaves the vector-memory and export counters free: vmcnt 63, expcnt 7,
// lgkmcnt 0.
constexpr int kWaitLgkm0 = 0xC07F;

// s_waitcnt for at most N outstanding vector-memory operations (6-bit
// vmcnt: low bits 3:0, high bits 15:14), leaving the export and LDS
// counters free.
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// K-loop issue plan, as 16-bit masks over the 16 MFMAs of a k step (bit n:
// after MFMA n): the 8 fragment reads of the next k step, the 8 direct loads
// of A two stages ahead over k steps 0..2, and the 8 of B two stages ahead in
// k step 3 (after the stage barrier, which frees its slot).  A wave stalls
// when the load path's queue is full and the four waves issue in step, so
// the loads of A are spread out.
constexpr int kReadMask = 0x00FF;
constexpr int kDmaA0 = 0x8800, kDmaA1 = 0x8888, kDmaA2 = 0x8800;
constexpr int kDmaB3 = 0xFF00;
static_assert(__builtin_popcount(kDmaA0) + __builtin_popcount(kDmaA1) +
                      __builtin_popcount(kDmaA2) == 8 &&
                  __builtin_popcount(kDmaB3) == 8 && __builtin_popcount(kReadMask) == 8,
              "eight loads of each operand and eight reads per k step");

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup barrier of the K loop.  __syncthreads() would also wait for every
// outstanding vector-memory operation, i.e. drain the direct-to-LDS loads of
// the later stages and leave no load in flight across the barrier; here the
// caller waits for exactly the stage it needs (vmcnt) and the memory clobber
// keeps the compiler from moving LDS accesses across the barrier.  The
// operand reads of the previous stage have completed by then: the MFMAs that
// consume them were issued before it.
__device__ __forceinline__ void stage_barrier() { asm volatile("s_barrier" ::: "memory"); }

// One 256x256 output tile: rows [mt*256, M) against column tile nt of Bm.
// HD (64 or 128) is the head size of the rotary epilogues (0 otherwise).
// EXT: the shapes and inputs beyond the plain case -- a ragged last column
// tile (N not a multiple of 256), cache sections that do not align with the
// 128-column waves (H*hd not a multiple of 128), a per-row second A buffer;
// the plain instantiation carries none of their per-lane tests (registers).
template <int EPI, bool GROUPED, int HD, bool EXT>
__device__ __forceinline__ void gemm_tile(const GP& p, char* smem, int layer, int mt, int nt,
                                          int M, const bf16* Bm) {
  // the wave index in a scalar register: LDS destinations of the direct
  // loads (M0) then need no read-back from a vector register
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = mt * BM;

  // ---- load assignment: DMA instruction j (0..7) of wave w fills the 1 KiB
  // of stage rows 8q .. 8q+7, q = w*8 + j; lane l -> row 8q + l/8, stored
  // position l%8, logical chunk (l%8) ^ ((row >> 1) & 7)
  // = (l%8) ^ ((4q + (l >> 4)) & 7).  A row's 128 bytes are one cache line.
  const int lrow = lane >> 3;
  const bf16* a_src[8];
  const bf16* b_src[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int q = wave * 8 + j;
    const int r = 8 * q + lrow;
    const int lchunk = (lane & 7) ^ ((4 * q + (lane >> 4)) & 7);
    int m = m0 + r;
    if (m >= M) m = m0;  // clamp: loaded, never stored
    const int arow = GROUPED ? (p.a_sorted ? m : p.srows[m]) : (p.a_rows ? p.a_rows[m] : m);
    const bf16* abase = (EXT && !GROUPED && p.a_sel && (p.a_sel[arow] & 1)) ? p.A2 : p.A;
    a_src[j] = abase + (int64_t)arow * p.lda + lchunk * 8;
    const bf16* bbase = Bm;
    int64_t brow;
    if (EPI == EPI_SWIGLU) {
      const int half = r >> 7, within = r & 127;
      bbase = within < 64 ? p.B : p.B2;
      brow = (int64_t)nt * 128 + half * 64 + (within & 63);
    } else {
      // a ragged last column tile re-reads the last row: computed, never stored
      brow = EXT ? min((int64_t)nt * BN + r, (int64_t)p.N - 1) : (int64_t)nt * BN + r;
    }
    b_src[j] = bbase + brow * p.ldb + lchunk * 8;
  }
  // Per-row inputs of the epilogue (row scale, residual row or cache slot,
  // rotary position) for the wave's 128 rows, two per lane: loaded here so
  // that their latency (two dependent loads for a cache slot) passes during
  // the K loop.
  float pre_sc[2];
  int pre_row[2], pre_pos[2];
  {
    constexpr bool kC = EPI == EPI_QKV || EPI == EPI_KV;
    const int secp = kC ? (nt * BN + wn * 128) / p.d_q : 0;
    const bool q_sec = EPI == EPI_QKV && secp == 0;
    const bool v_sec = EPI == EPI_QKV ? secp == 2 : (EPI == EPI_KV && secp == 1);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int mc = min(m0 + wm * 128 + lane + 64 * h, M - 1);   // clamped: never stored
      pre_sc[h] = p.row_scale ? p.row_scale[mc] : 1.0f;
      pre_row[h] = 0;
      pre_pos[h] = 0;
      if (EPI == EPI_RESID) {
        pre_row[h] = p.rows[mc];
      } else if (kC) {
        const int row = GROUPED ? p.srows[mc] : p.rows[mc];
        pre_row[h] = (q_sec && p.d_q % 128 == 0) ? 0 : (p.slot ? p.slot[row] : row);
        pre_pos[h] = (v_sec || !p.rope_cos) ? 0 : p.pos[row];
      }
    }
  }
  // Ring of kSlots one-operand slots: A of stage k in slot 2k mod 5, B of
  // stage k in slot 2k+1 mod 5.  DMA instruction j (0..7) of an operand.
  auto slot = [&](int u) { return smem + (u % kSlots) * kStageBytes; };
  auto issue_a = [&](int k, int u, int j) {
    dma16(a_src[j] + k * BK, slot(u) + (wave * 8 + j) * 1024);
  };
  auto issue_b = [&](int k, int u, int j) {
    dma16(b_src[j] + k * BK, slot(u) + (wave * 8 + j) * 1024);
  };

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  // MFMA operand addresses: block i row R = w*128 + i*32 + lane%32; logical
  // chunk 2*ks + lane/32 (k step ks = 0..3) stored at chunk ^ ((R >> 1) & 7),
  // and the block offsets are multiples of 32, so the position is
  // chunk ^ ((lane >> 1) & 7).
  const int rA = wm * 128 + (lane & 31);
  const int rB = wn * 128 + (lane & 31);
  const int swz = (lane >> 1) & 7;
  const int KT = p.K / BK;
  // Fragment reads from a slot known at compile time: win[o][w][ks] + a
  // constant, with window w (64 KiB of the ring) plus the lane's offset of k
  // step ks in block 0 of operand o (0 = A, 1 = B); the slot within the
  // window and the block (i * 4 KiB) fit the 16-bit offset of ds_read, so a
  // read takes no address arithmetic.
  lds_char_t* win[2][3][4];
#pragma unroll
  for (int o = 0; o < 2; ++o)
#pragma unroll
    for (int w = 0; w < 3; ++w)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        win[o][w][ks] = (lds_char_t*)smem + w * 65536 +
                        ((o ? rB : rA) * 8 + ((2 * ks + (lane >> 5)) ^ swz)) * 16;
  // Re-defines the bases (no instruction): otherwise the compiler hoists
  // the addresses derived for every slot, operand and k step out of the
  // loop, into registers of their own.
  auto refresh = [&]() {
#pragma unroll
    for (int o = 0; o < 2; ++o)
#pragma unroll
      for (int w = 0; w < 3; ++w)
        asm volatile("" : "+v"(win[o][w][0]), "+v"(win[o][w][1]), "+v"(win[o][w][2]),
                     "+v"(win[o][w][3]));
  };
  // Fragment n (0..7: A block n/2 for even n, B block n/2 for odd n) of k
  // step ks from slots uA / uB, compile-time slots (fixed) or any slot
  // (run-time address arithmetic).
  auto frag_fixed = [&](int uA, int uB, int ks, int n, bf16x8_t (&a)[4], bf16x8_t (&b)[4]) {
    const int i = n >> 1;
    uA %= kSlots;
    uB %= kSlots;
    if (n & 1)
      b[i] = *reinterpret_cast<const lds_bf16x8_t*>(win[1][uB >> 1][ks] + (uB & 1) * kStageBytes +
                                                    i * 4096);
    else
      a[i] = *reinterpret_cast<const lds_bf16x8_t*>(win[0][uA >> 1][ks] + (uA & 1) * kStageBytes +
                                                    i * 4096);
  };
  auto frag_any = [&](int uA, int uB, int ks, int n, bf16x8_t (&a)[4], bf16x8_t (&b)[4]) {
    const int ch = (2 * ks + (lane >> 5)) ^ swz;
    const int i = n >> 1;
    if (n & 1)
      b[i] = *reinterpret_cast<const lds_bf16x8_t*>((lds_char_t*)slot(uB) +
                                                    ((rB + i * 32) * 8 + ch) * 16);
    else
      a[i] = *reinterpret_cast<const lds_bf16x8_t*>((lds_char_t*)slot(uA) +
                                                    ((rA + i * 32) * 8 + ch) * 16);
  };
  // One k step: 16 MFMAs on (a, b).  After MFMA n, read(r) issues fragment
  // r of the next k step when bit n of RMASK is set, and dma(d) issues DMA
  // instruction d0 + (number of DMAs already issued in this step) when bit
  // n of DMASK is set, so that every non-MFMA instruction issues while the
  // matrix core has work queued.  The masks are compile-time constants: a
  // branch between MFMAs costs an instruction-fetch bubble.
  auto kstep = [&](const bf16x8_t (&a)[4], const bf16x8_t (&b)[4], auto&& read, auto&& dma,
                   auto rmask, auto dmask, int d0) {
    constexpr int RM = decltype(rmask)::value, DM = decltype(dmask)::value;
#pragma unroll
    for (int n = 0; n < 16; ++n) {
      const int i = n >> 2, j = n & 3;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      if ((RM >> n) & 1) read(__builtin_popcount(RM & ((1 << n) - 1)));
      if ((DM >> n) & 1) dma(d0 + __builtin_popcount(DM & ((1 << n) - 1)));
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using Reads = std::integral_constant<int, kReadMask>;
  using A0 = std::integral_constant<int, kDmaA0>;
  using A1 = std::integral_constant<int, kDmaA1>;
  using A2 = std::integral_constant<int, kDmaA2>;
  using B3 = std::integral_constant<int, kDmaB3>;
  constexpr int kA01 = __builtin_popcount(kDmaA0) + __builtin_popcount(kDmaA1);

  // K loop over a 5-slot ring (A of stage k in slot 2k mod 5, B in 2k+1
  // mod 5).  At the top of iteration kt stage kt has landed and is visible
  // to every wave, A_kt+1 and B_kt+1 are in flight, and the fragments of
  // stage kt's first k step were read just before.  A slot is refilled as
  // soon as a barrier retires its last reads: A_kt+2 goes into the slot of
  // B_kt-1 during k steps 0..2, and B_kt+2 into the slot of A_kt right after
  // this iteration's barrier, so each stage has one to two iterations of
  // MFMA work to land.  Before each k step, the reads issued during the
  // previous one are waited for; at most 8 LDS reads are ever outstanding
  // (the 4-bit lgkm counter cannot express more).  The wait for stage kt+1
  // (only A_kt+2, issued last, may stay outstanding) and the barrier, which
  // publishes stage kt+1 and retires every read of stage kt, come before the
  // last k step, whose 16 MFMAs then cover the reads of stage kt+1's first
  // fragments.
  //
  // Every iteration issues the same loads: past the last stage the stage
  // index is clamped, so the last two iterations refill free slots with
  // data that is never read (two stages of extra L2 traffic per tile) and
  // the body has no conditional code.  The loop runs in groups of five, the
  // ring's period, in which every slot is a compile-time constant; the
  // KT mod 5 iterations before them take the same body with run-time slots.
  const int kLast = KT - 1;
  // stage k's slots are shifted by sh so that the groups of five, which
  // follow the KT mod 5 iterations with run-time slots, start at phase 0
  const int sh = (kSlots - KT % kSlots) % kSlots;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    issue_a(0, 2 * sh, j);
    issue_b(0, 2 * sh + 1, j);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    issue_a(min(1, kLast), 2 * sh + 2, j);
    issue_b(min(1, kLast), 2 * sh + 3, j);
  }
  wait_vm<16>();
  stage_barrier();
  bf16x8_t fa[4], fb[4], ga[4], gb[4];
#pragma unroll
  for (int n = 0; n < 8; ++n) frag_any(2 * sh, 2 * sh + 1, 0, n, fa, fb);
  // iteration kt, with P = (kt + sh) mod 5 (a compile-time constant when FIXED)
  auto iteration = [&](int kt, int P, auto fixed) {
    constexpr bool kFixed = decltype(fixed)::value;
    auto frag = [&](int uA, int uB, int ks, int n, bf16x8_t (&a)[4], bf16x8_t (&b)[4]) {
      if constexpr (kFixed) frag_fixed(uA, uB, ks, n, a, b);
      else frag_any(uA, uB, ks, n, a, b);
    };
    const int kd = min(kt + 2, kLast);
    const int uA = 2 * P, uB = 2 * P + 1;
    auto dma_a = [&](int j) { issue_a(kd, 2 * P + 4, j); };
    if constexpr (kFixed) refresh();
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_sched_barrier(0);
    kstep(fa, fb, [&](int n) { frag(uA, uB, 1, n, ga, gb); }, dma_a, Reads{}, A0{}, 0);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_sched_barrier(0);
    kstep(ga, gb, [&](int n) { frag(uA, uB, 2, n, fa, fb); }, dma_a, Reads{}, A1{},
          __builtin_popcount(kDmaA0));
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_sched_barrier(0);
    kstep(fa, fb, [&](int n) { frag(uA, uB, 3, n, ga, gb); }, dma_a, Reads{}, A2{}, kA01);
    // every read of stage kt has completed: wait for stage kt+1 (A_kt+2,
    // issued last, may stay outstanding), publish it, retire stage kt's slots
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_sched_barrier(0);
    wait_vm<8>();
    stage_barrier();
    // after the last stage this reads stale but valid LDS
    kstep(ga, gb, [&](int n) { frag(uA + 2, uB + 2, 0, n, fa, fb); },
          [&](int j) { issue_b(kd, 2 * P, j); }, Reads{}, B3{}, 0);
  };
  using Fixed = std::true_type;
  using Any = std::false_type;
  const int r = KT % kSlots;
  int kt = 0;
  for (; kt < r; ++kt) iteration(kt, (kt + sh) % kSlots, Any{});
  for (; kt < KT; kt += kSlots) {
    iteration(kt, 0, Fixed{});
    iteration(kt + 1, 1, Fixed{});
    iteration(kt + 2, 2, Fixed{});
    iteration(kt + 3, 3, Fixed{});
    iteration(kt + 4, 4, Fixed{});
  }
  wait_dma();   // the clamped loads of the last iterations land before LDS is reused
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  stage_barrier();   // every wave is done with the ring; LDS is reused below

  // ---- epilogue, staged through LDS 32 rows at a time.  Lane holds column
  // (lane & 31) of each 32x32 block and rows 8*(v/4) + 4*(lane/32) + v%4,
  // v = 0..15.  Block i of the wave (32 rows x its 128 columns, f32) is
  // written to the wave's LDS area with a row stride of kEpiStride floats
  // (the two row groups of a write then fall on disjoint banks), then read
  // back as 4 consecutive columns per lane, so every global load and store
  // of the epilogue covers whole rows: 32 lanes x 8 bytes = one 256-byte row
  // of 128 bf16 columns.  The per-row inputs (scale, residual row or cache
  // slot and position) of the wave's 128 rows are gathered into LDS first,
  // two memory latencies per tile instead of one per store round.
  float* stg = reinterpret_cast<float*>(smem + wave * kEpiWaveBytes);
  float* msc = reinterpret_cast<float*>(smem + 4 * kEpiWaveBytes + wave * kEpiMetaBytes);
  int* mrow = reinterpret_cast<int*>(msc + 128);   // residual row / cache slot
  int* mpos = mrow + 128;                          // rotary position
  const int col_l = lane & 31;
  const int row_q = 4 * (lane >> 5);
  const int c4 = (lane & 31) * 4;         // first of the lane's 4 columns (wave space)
  const int nw = nt * BN + wn * 128;      // first output column of this wave
  // grouped: layer r's bias; a ragged column tile's waves past N store
  // nothing (SwiGLU tiles are never ragged: 128 outputs of N per tile)
  const bf16* bias = GROUPED && EXT && p.bias ? p.bias + (int64_t)(layer - 1) * p.bias_layer_stride
                                       : p.bias;
  const bool wave_out = EXT && EPI != EPI_SWIGLU && nw >= p.N;
  constexpr bool kCache = EPI == EPI_QKV || EPI == EPI_KV;
  const int sec = kCache ? nw / p.d_q : 0;    // QKV: 0 q, 1 k, 2 v;  KV: 0 k, 1 v
  const bool is_q = EPI == EPI_QKV && sec == 0;
  const bool is_v = EPI == EPI_QKV ? sec == 2 : (EPI == EPI_KV && sec == 1);
  const int cbase = nw - sec * p.d_q;         // column within the section
  constexpr int hd = HD > 0 ? HD : 128, half = hd >> 1;
  // destination of the QKV / KV epilogues: Q rows by compact index, K and V
  // rows by cache slot (in layer r's cache for the grouped variant)
  bf16* sec_dst = nullptr;
  if (kCache) {
    if (is_q) {
      sec_dst = p.q_out;
    } else {
      sec_dst = is_v ? p.v_cache : p.k_cache;
      if (GROUPED) sec_dst += (int64_t)(layer - 1) * p.cache_layer_stride;
    }
    sec_dst += cbase;
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int lr = lane + 64 * h;
    msc[lr] = pre_sc[h];
    if (EPI == EPI_RESID || kCache) mrow[lr] = pre_row[h];
    if (kCache) mpos[lr] = pre_pos[h];
  }
  // one 32-row block; the block index is a compile-time constant (an
  // accumulator indexed at run time would move the whole tile to scratch)
  auto block = [&](auto ic) {
    constexpr int i = decltype(ic)::value;
    const int mb = m0 + wm * 128 + i * 32;   // first row of the block
    if (mb >= M || wave_out) return;          // rows past M / columns past N
    if constexpr (EPI == EPI_SWIGLU) {
      // Gate (blocks j = 0, 1) and up (j = 2, 3) of an output column sit in
      // the same lane, so h = silu(g) * u is formed in registers; lanes 2k
      // and 2k+1 hold adjacent columns and swap one value (DPP), so the even
      // lane holds row v and the odd lane row v+1 of a pair of columns as
      // one 4-byte bf16 pair.  The pairs go to LDS (32 rows x 128 bytes; two
      // rows fill the 64 banks) and come back as 16-byte row segments: four
      // full-row stores per block instead of 32 narrow ones.
      float sc[16];
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const float4 t = *reinterpret_cast<const float4*>(msc + i * 32 + 8 * g4 + row_q);
        sc[4 * g4 + 0] = t.x; sc[4 * g4 + 1] = t.y; sc[4 * g4 + 2] = t.z; sc[4 * g4 + 3] = t.w;
      }
      const bool odd = lane & 1;
      char* sb = reinterpret_cast<char*>(stg);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int v0 = 2 * t, v1 = 2 * t + 1;
          const float h0 = silu(acc[i][j][v0] * sc[v0]) * (acc[i][j + 2][v0] * sc[v0]);
          const float h1 = silu(acc[i][j][v1] * sc[v1]) * (acc[i][j + 2][v1] * sc[v1]);
          // quad_perm [1,0,3,2]: exchange with the neighbouring lane
          const float y = __int_as_float(__builtin_amdgcn_mov_dpp(
              __float_as_int(odd ? h0 : h1), 0xB1, 0xF, 0xF, false));
          const uint32_t w = odd ? pack_bf16x2(y, h1) : pack_bf16x2(h0, y);
          const int lr = 8 * (v0 >> 2) + row_q + (v0 & 3) + (odd ? 1 : 0);
          *reinterpret_cast<uint32_t*>(sb + lr * 128 + j * 64 + (col_l & ~1) * 2) = w;
        }
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      __builtin_amdgcn_wave_barrier();
      const bool full = mb + 32 <= M;
      bf16* cb = reinterpret_cast<bf16*>(p.C) + nt * 128 + wn * 64 + (lane & 7) * 8;
      uint4 seg[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        seg[q] = *reinterpret_cast<const uint4*>(sb + (8 * q + (lane >> 3)) * 128 + (lane & 7) * 16);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m = mb + 8 * q + (lane >> 3);
        if (full || m < M) *reinterpret_cast<uint4*>(cb + (int64_t)m * p.ldc) = seg[q];
      }
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);   // reads done before the next block's writes
      __builtin_amdgcn_wave_barrier();
      return;
    }
    if constexpr (kCache) {
      if (!p.bias) {   // wave-uniform: the decoder's QKV and the KV generation
        // The wave's 128 columns are whole heads, so the rotary partner of a
        // column (c ^ hd/2) sits in the same lane, hd/64 blocks away: RoPE
        // runs on the accumulators.  Positions come from the gathered
        // per-row inputs and the cos/sin values of the block's 16 rows per
        // lane are loaded at once (one memory latency per block).  Results
        // leave as in the SwiGLU path: bf16 pairs (DPP lane swap) to LDS,
        // 32 rows x 256 bytes, each row's four 64-byte segments permuted by
        // (row & 1) | ((row >> 2) & 1) << 1 so the four row groups of a
        // write fall on distinct banks, read back as 16-byte row segments
        // and stored as whole 256-byte rows of the destination.
        constexpr int kPair = hd / 64;          // block distance of rotary partners
        constexpr int kTab = hd == 128 ? 2 : 1; // table columns per lane and row
        const bool rope = !is_v && p.rope_cos;  // wave-uniform
        float sc[16];
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const float4 t = *reinterpret_cast<const float4*>(msc + i * 32 + 8 * g4 + row_q);
          sc[4 * g4 + 0] = t.x; sc[4 * g4 + 1] = t.y; sc[4 * g4 + 2] = t.z; sc[4 * g4 + 3] = t.w;
        }
        float cv[16][kTab], sv[16][kTab];
        if (rope) {
          int ps[16];
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int4 t = *reinterpret_cast<const int4*>(mpos + i * 32 + 8 * g4 + row_q);
            ps[4 * g4 + 0] = t.x; ps[4 * g4 + 1] = t.y; ps[4 * g4 + 2] = t.z; ps[4 * g4 + 3] = t.w;
          }
#pragma unroll
          for (int v = 0; v < 16; ++v)
#pragma unroll
            for (int u = 0; u < kTab; ++u) {
              const int64_t t = (int64_t)ps[v] * half + u * 32 + col_l;
              cv[v][u] = p.rope_cos[t];
              sv[v][u] = p.rope_sin[t];
            }
        }
        // output of column block j, row v of the lane
        auto out = [&](int j, int v) {
          const float x = acc[i][j][v] * sc[v];
          if (!rope) return x;
          const float y = acc[i][j ^ kPair][v] * sc[v];
          const int u = hd == 128 ? (j & 1) : 0;
          const bool first = hd == 128 ? j < 2 : (j & 1) == 0;   // column < hd/2
          return first ? x * cv[v][u] - y * sv[v][u] : x * cv[v][u] + y * sv[v][u];
        };
        // Lanes 2k, 2k+1 hold adjacent columns.  Each packs its rows v0, v1
        // as one bf16 pair, the pairs are swapped (DPP quad_perm [1,0,3,2])
        // and one byte permute forms row v0 (even lane) or row v1 (odd
        // lane) of the two columns.
        const bool odd = lane & 1;
        const uint32_t psel = odd ? 0x03020706u : 0x05040100u;
        char* sb = reinterpret_cast<char*>(stg);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const int v0 = 2 * t, v1 = 2 * t + 1;
            const uint32_t own = pack_bf16x2(out(j, v0), out(j, v1));
            const uint32_t nbr = (uint32_t)__builtin_amdgcn_mov_dpp((int)own, 0xB1, 0xF, 0xF, false);
            const uint32_t w = __builtin_amdgcn_perm(nbr, own, psel);
            const int lr = 8 * (v0 >> 2) + row_q + (v0 & 3) + (odd ? 1 : 0);
            const int g = (lr & 1) | (((lr >> 2) & 1) << 1);
            *reinterpret_cast<uint32_t*>(sb + lr * 256 + ((j ^ g) << 6) + (col_l & ~1) * 2) = w;
          }
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        __builtin_amdgcn_wave_barrier();
        const bool full = mb + 32 <= M;
        const int sg = lane & 15;
        typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
        u32x4_t seg[8];
        int drow[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int R = 4 * q + (lane >> 4);
          const int g = (R & 1) | (((R >> 2) & 1) << 1);
          seg[q] = *reinterpret_cast<const u32x4_t*>(sb + R * 256 + (((sg >> 2) ^ g) << 6) +
                                                     (sg & 3) * 16);
          drow[q] = is_q ? mb + R : mrow[i * 32 + R];
        }
        // cache rows are streamed out (not read again while cached); Q rows
        // are read by the attention that follows
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int m = mb + 4 * q + (lane >> 4);
          u32x4_t* dst = reinterpret_cast<u32x4_t*>(sec_dst + (int64_t)drow[q] * p.d_q + sg * 8);
          if (full || m < M) {
            if (is_q) *dst = seg[q];
            else __builtin_nontemporal_store(seg[q], dst);
          }
        }
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);   // reads done before the next block's writes
        __builtin_amdgcn_wave_barrier();
        return;
      }
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int lr = 8 * (v >> 2) + row_q + (v & 3);
#pragma unroll
      for (int j = 0; j < 4; ++j) stg[lr * kEpiStride + j * 32 + col_l] = acc[i][j][v];
    }
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_wave_barrier();
    if constexpr (EPI == EPI_RESID || EPI == EPI_STORE || EPI == EPI_GELU ||
                  EPI == EPI_GELU_TANH) {
      if (EPI != EPI_STORE || !p.c_f32) {   // wave-uniform
        // Row-segment form: 16 lanes per row, 8 consecutive columns per lane
        // (two 16-byte LDS reads of the staged f32 row), so the residual
        // segment is one 16-byte load and the result one 16-byte store; the
        // 8 residual loads of a block are issued together (one memory
        // latency per block).  The sum is rounded to bf16 once.
        const bool full = mb + 32 <= M;
        const int sg = lane & 15;
        const int col = nw + 8 * sg;
        const bool col_in = !EXT || col < p.N;   // N is a multiple of 64: whole 8-column segments
        int drow[8];
        float scv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int R = 4 * q + (lane >> 4);
          drow[q] = EPI == EPI_RESID ? mrow[i * 32 + R] : mb + R;
          scv[q] = msc[i * 32 + R];
        }
        uint4 rres[8];
        if constexpr (EPI == EPI_RESID) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const int m = mb + 4 * q + (lane >> 4);
            rres[q] = ((full || m < M) && col_in) ? *reinterpret_cast<const uint4*>(
                                            reinterpret_cast<const bf16*>(p.resid) +
                                            (int64_t)drow[q] * p.ldc + col)
                                      : make_uint4(0, 0, 0, 0);
          }
        }
        const float4 b0 = bias4(col_in ? bias : nullptr, col);
        const float4 b1 = bias4(col_in ? bias : nullptr, col + 4);
        const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int R = 4 * q + (lane >> 4);
          const int m = mb + R;
          const float4 f0 = *reinterpret_cast<const float4*>(stg + R * kEpiStride + 8 * sg);
          const float4 f1 = *reinterpret_cast<const float4*>(stg + R * kEpiStride + 8 * sg + 4);
          const float f[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
          float x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            x[e] = f[e] * scv[q] + bv[e];
            if constexpr (EPI == EPI_GELU) x[e] = gelu_erf(x[e]);
            if constexpr (EPI == EPI_GELU_TANH) x[e] = gelu_tanh(x[e]);
          }
          if constexpr (EPI == EPI_RESID) {
            const uint32_t rw[4] = {rres[q].x, rres[q].y, rres[q].z, rres[q].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              x[2 * e] += __uint_as_float(rw[e] << 16);
              x[2 * e + 1] += __uint_as_float(rw[e] & 0xffff0000u);
            }
          }
          const uint4 o = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]),
                                     pack_bf16x2(x[4], x[5]), pack_bf16x2(x[6], x[7]));
          if ((full || m < M) && col_in)
            *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C) + (int64_t)drow[q] * p.ldc +
                                      col) = o;
        }
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);   // reads done before the next block's writes
        __builtin_amdgcn_wave_barrier();
        return;
      }
    }
    // Each block is emitted in phases: all LDS reads of a group of rounds
    // into registers, then the global loads they index, then arithmetic and
    // stores (the stores go through generic pointers, which the compiler
    // must otherwise keep ordered before later LDS reads).  Rows past M exist
    // only in the last block of a ragged tile; full blocks take the variant
    // without the per-row store check.
    auto emit = [&](auto check) {
      constexpr bool kCheck = decltype(check)::value;
      if (EPI == EPI_SWIGLU) {
        // 64 outputs per row (gate columns 0..63 of the wave, up columns
        // 64..127): 16 lanes per row, 4 rows per round, 8 rounds
        const int c = (lane & 15) * 4;
        float4 g[8], u[8];
        float sc[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const int lr = 4 * r + (lane >> 4);
          g[r] = *reinterpret_cast<const float4*>(stg + lr * kEpiStride + c);
          u[r] = *reinterpret_cast<const float4*>(stg + lr * kEpiStride + 64 + c);
          sc[r] = msc[i * 32 + lr];
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const int m = mb + 4 * r + (lane >> 4);
          bf16x4_t o;
          o[0] = f2bf(silu(g[r].x * sc[r]) * (u[r].x * sc[r]));
          o[1] = f2bf(silu(g[r].y * sc[r]) * (u[r].y * sc[r]));
          o[2] = f2bf(silu(g[r].z * sc[r]) * (u[r].z * sc[r]));
          o[3] = f2bf(silu(g[r].w * sc[r]) * (u[r].w * sc[r]));
          if (!kCheck || m < M)
            *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + (int64_t)m * p.ldc +
                                         nt * 128 + wn * 64 + c) = o;
        }
      } else {
        // 2 rows per round (32 lanes x 4 columns each), 16 rounds in groups of
        // G (4 for the rotary epilogues, whose rounds hold 4 float4 each)
        constexpr bool kRope = EPI == EPI_QKV || EPI == EPI_KV;
        constexpr int G = kRope ? 4 : 8;
        const bool rope = kRope && !is_v && p.rope_cos;   // wave-uniform
        const bool col_in = !EXT || nw + c4 < p.N;        // N is a multiple of 4
        const float4 bx = bias4(col_in ? bias : nullptr, nw + c4);
        const float4 by = rope ? bias4(bias, nw + (c4 ^ half)) : bx;
        // a wave's 128 columns lie in one section (Q, K or V) when d_q is a
        // multiple of 128; otherwise (no RoPE then) each lane finds its own
        const bool sec_wave = !EXT || p.d_q % 128 == 0;     // wave-uniform
#pragma unroll
        for (int hh = 0; hh < 16 / G; ++hh) {
          float4 x4[G], y4[G], cs[G], sn[G];
          float sc[G];
          int mr[G], mp[G];
          bf16x4_t rv[G];
#pragma unroll
          for (int r = 0; r < G; ++r) {
            const int lr = 2 * (G * hh + r) + (lane >> 5);
            x4[r] = *reinterpret_cast<const float4*>(stg + lr * kEpiStride + c4);
            if (rope)
              y4[r] = *reinterpret_cast<const float4*>(stg + lr * kEpiStride + (c4 ^ half));
            sc[r] = msc[i * 32 + lr];
            mr[r] = mrow[i * 32 + lr];
            mp[r] = mpos[i * 32 + lr];
          }
#pragma unroll
          for (int r = 0; r < G; ++r) {
            if (EPI == EPI_RESID && col_in)
              rv[r] = *reinterpret_cast<const bf16x4_t*>(p.resid + (int64_t)mr[r] * p.ldc + nw + c4);
            if (rope) {
              const int c = (cbase + c4) & (hd - 1);
              const int64_t t = (int64_t)mp[r] * half + (c & (half - 1));
              cs[r] = *reinterpret_cast<const float4*>(p.rope_cos + t);
              sn[r] = *reinterpret_cast<const float4*>(p.rope_sin + t);
            }
          }
#pragma unroll
          for (int r = 0; r < G; ++r) {
            const int m = mb + 2 * (G * hh + r) + (lane >> 5);
            const float x[4] = {x4[r].x * sc[r] + bx.x, x4[r].y * sc[r] + bx.y,
                                x4[r].z * sc[r] + bx.z, x4[r].w * sc[r] + bx.w};
            bf16x4_t o;
            if (EPI == EPI_GELU || EPI == EPI_GELU_TANH) {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                o[e] = f2bf(EPI == EPI_GELU ? gelu_erf(x[e]) : gelu_tanh(x[e]));
              if ((!kCheck || m < M) && col_in)
                *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + (int64_t)m * p.ldc +
                                             nw + c4) = o;
            } else if (EPI == EPI_STORE) {
              const int64_t off = (int64_t)m * p.ldc + nw + c4;
              if ((!kCheck || m < M) && col_in) {
                if (p.c_f32) {
                  *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.C) + off) =
                      make_float4(x[0], x[1], x[2], x[3]);
                } else {
#pragma unroll
                  for (int e = 0; e < 4; ++e) o[e] = f2bf(x[e]);
                  *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + off) = o;
                }
              }
            } else if (EPI == EPI_RESID) {
#pragma unroll
              for (int e = 0; e < 4; ++e) o[e] = f2bf(x[e] + bf2f(rv[r][e]));
              if ((!kCheck || m < M) && col_in)
                *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) +
                                             (int64_t)mr[r] * p.ldc + nw + c4) = o;
            } else {  // EPI_QKV / EPI_KV
              if (!rope) {
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = f2bf(x[e]);
              } else {
                // rotate-half RoPE: column c pairs with c +- hd/2 of the same head
                const float y[4] = {y4[r].x * sc[r] + by.x, y4[r].y * sc[r] + by.y,
                                    y4[r].z * sc[r] + by.z, y4[r].w * sc[r] + by.w};
                const int c = (cbase + c4) & (hd - 1);   // column within the head
                const float cv[4] = {cs[r].x, cs[r].y, cs[r].z, cs[r].w};
                const float sv[4] = {sn[r].x, sn[r].y, sn[r].z, sn[r].w};
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  o[e] = f2bf(c < half ? x[e] * cv[e] - y[e] * sv[e] : x[e] * cv[e] + y[e] * sv[e]);
              }
              if (rope || sec_wave) {
                const int64_t drow = is_q ? (int64_t)m : (int64_t)mr[r];
                if ((!kCheck || m < M) && col_in)
                  *reinterpret_cast<bf16x4_t*>(sec_dst + drow * p.d_q + c4) = o;
              } else {
                const int secl = (nw + c4) / p.d_q;
                const bool lq = EPI == EPI_QKV && secl == 0;
                const bool lv = EPI == EPI_QKV ? secl == 2 : (EPI == EPI_KV && secl == 1);
                bf16* ldst = lq ? p.q_out
                                : (lv ? p.v_cache : p.k_cache) +
                                      (GROUPED ? (int64_t)(layer - 1) * p.cache_layer_stride : 0);
                const int64_t drow = lq ? (int64_t)m : (int64_t)mr[r];
                if ((!kCheck || m < M) && col_in)
                  *reinterpret_cast<bf16x4_t*>(ldst + drow * p.d_q + nw + c4 - secl * p.d_q) = o;
              }
            }
          }
        }
      }
    };
    if (mb + 32 <= M) emit(std::false_type{});
    else emit(std::true_type{});
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);   // block reads done before the next block's writes
    __builtin_amdgcn_wave_barrier();
  };
  block(std::integral_constant<int, 0>{});
  block(std::integral_constant<int, 1>{});
  block(std::integral_constant<int, 2>{});
  block(std::integral_constant<int, 3>{});
}

// XCD-aware tile order (see the header comment).
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int* mt, int* nt) {
  const int T = tiles_m * tiles_n;
  int t = bid;
  if ((T & 7) == 0) t = (bid & 7) * (T >> 3) + (bid >> 3);
  constexpr int G = 8;  // row tiles per raster group
  const int gsz = G * tiles_n;
  const int g = t / gsz, r = t - g * gsz;
  const int rows_in_g = min(G, tiles_m - g * G);
  *mt = g * G + r % rows_in_g;
  *nt = r / rows_in_g;
}

// The grid is sized for M_max; the tiles are numbered over the rows that are
// actually active (device count), so when tokens exit the remaining tiles
// still spread over all XCDs and the surplus workgroups return at once.
template <int EPI, int HD, bool EXT>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(GP p) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int M = p.M_dev ? min(*p.M_dev, p.M_max) : p.M_max;
  const int tiles_m = (M + BM - 1) / BM;
  if ((int)blockIdx.x >= tiles_m * p.tiles_n) return;
  int mt, nt;
  tile_of(blockIdx.x, tiles_m, p.tiles_n, &mt, &nt);
  gemm_tile<EPI, false, HD, EXT>(p, smem, 0, mt, nt, M, p.B);
}

// Grouped GEMM of the KV generation: one workgroup per item of the
// device-built list of (layer, row tile) items times the column tiles,
// rastered in groups of 8 row tiles.  Workgroup ids go to the 8 XCDs
// round-robin, so XCD x takes the x-th contiguous eighth of the item list and
// the tiles running together on an XCD share one layer's weight slices in its
// L2; ids past the device-built count return at once.  (A persistent form
// that took items from per-XCD counters kept the loop's state in registers
// and spilled 196 bytes per lane around the K loop; one item per workgroup
// compiles as the plain GEMM does, without scratch, and runs 2 % faster.)
template <int HD, bool EXT>
__global__ __launch_bounds__(kThreads, 1) void gemm_kv_flat_kernel(GP p) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int n_work = *p.n_work;
  const int total = n_work * p.tiles_n;
  const int chunk = (total + 7) >> 3;
  const int t = (int)(blockIdx.x & 7) * chunk + (int)(blockIdx.x >> 3);
  if ((int)(blockIdx.x >> 3) >= chunk || t >= total) return;
  constexpr int G = 8;
  const int gsz = G * p.tiles_n;
  const int g = t / gsz, r = t - g * gsz;
  const int rows_in_g = min(G, n_work - g * G);
  const int w = g * G + r % rows_in_g, nt = r / rows_in_g;
  const int packed = p.work[w];
  const int layer = packed >> 16, mt = packed & 0xffff;
  gemm_tile<EPI_KV, true, HD, EXT>(p, smem, layer, mt, nt, p.grp_m[layer],
                                   p.B + (int64_t)(layer - 1) * p.b_layer_stride);
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
      if (m >= M) m = m0;
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

// Element-wise epilogue over the f32 scratch T[m][n] (n < n_out), after the
// per-row scale.
__global__ void epilogue_f32_kernel(int epi, int M_max, const int32_t* M_dev, int n_out,
                                    const float* __restrict__ T, int64_t ldt, GP p) {
  const int M = M_dev ? min(*M_dev, M_max) : M_max;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int m = (int)(idx / n_out), n = (int)(idx % n_out);
  if (m >= M) return;
  const float sc = p.row_scale ? p.row_scale[m] : 1.0f;
  const float* t = T + (int64_t)m * ldt;
  float* C = reinterpret_cast<float*>(p.C);
  if (epi == EPI_STORE) {
    C[(int64_t)m * p.ldc + n] = t[n] * sc;
  } else if (epi == EPI_RESID) {
    const int64_t row = p.rows[m];
    C[row * p.ldc + n] = reinterpret_cast<const float*>(p.resid)[row * p.ldc + n] + t[n] * sc;
  } else if (epi == EPI_SWIGLU) {
    C[(int64_t)m * p.ldc + n] = silu(t[n] * sc) * (t[p.N + n] * sc);
  } else {  // EPI_QKV
    const int sec = n / p.d_q, cin = n - sec * p.d_q;
    const int row = p.rows[m];
    float* dst;
    if (sec == 0) dst = reinterpret_cast<float*>(p.q_out) + (int64_t)m * p.d_q;
    else dst = reinterpret_cast<float*>(sec == 1 ? p.k_cache : p.v_cache) + (int64_t)p.slot[row] * p.d_q;
    if (sec == 2) {
      dst[cin] = t[n] * sc;
    } else {
      const int hd = p.head_dim, half = hd / 2;
      const int c = cin % hd, kk = c % half;
      const int ps = p.pos[row];
      const float cs = p.rope_cos[(int64_t)ps * half + kk], sn = p.rope_sin[(int64_t)ps * half + kk];
      const float x = t[n] * sc;
      const float y = (c < half ? t[n + half] : t[n - half]) * sc;
      dst[cin] = c < half ? x * cs - y * sn : x * cs + y * sn;
    }
  }
}

// Sets the 128 KiB dynamic-LDS limit of a kernel once per process.
adept_status allow_lds(const void* kernel, bool* done, const char* what) {
  if (*done) return ADEPT_OK;
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes) !=
      hipSuccess)
    return launch_status(what);
  *done = true;
  return ADEPT_OK;
}

template <int EPI, int HD, bool EXT>
adept_status launch_bf16_x(const GP& p, hipStream_t s, const char* name) {
  static bool attr_set = false;
  ADEPT_TRY(allow_lds((const void*)gemm_bf16_kernel<EPI, HD, EXT>, &attr_set,
                      "gemm_bf16 LDS limit"));
  {
    TimedLaunch tl(name ? name : "gemm_bf16", s);
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI, HD, EXT>), dim3(p.tiles_m * p.tiles_n),
                       dim3(kThreads), kLdsBytes, s, p);
  }
  return launch_status("gemm_bf16");
}

// the extended instantiation only where the shape or the inputs need it
bool needs_ext(const GP& p, int epi) {
  return (epi != EPI_SWIGLU && p.N % BN != 0) ||
         ((epi == EPI_QKV || epi == EPI_KV) && p.d_q % 128 != 0) || p.a_sel != nullptr;
}

template <int EPI, int HD>
adept_status launch_bf16(const GP& p, hipStream_t s, const char* name) {
  return needs_ext(p, EPI) ? launch_bf16_x<EPI, HD, true>(p, s, name)
                           : launch_bf16_x<EPI, HD, false>(p, s, name);
}

// ---------------------------------------------------------------------------
// Skinny path (at most 64 rows: decode).  The weights are streamed from HBM
// once; M is too small for the 256x256 tile to give the chip enough
// workgroups.  The work is a flattened space of units: a unit is one
// 64-column tile of the partial space (N columns, or the
// F gate columns followed by the F up columns for SWIGLU) times one 64-deep
// k step.  The units are cut into G equal contiguous ranges, one per
// workgroup (stream-K), so that every workgroup streams the same number of
// weight bytes and the grid is one even wave of about two workgroups per CU;
// a range is never longer than a tile's k extent, so it covers at most two
// tiles (two segments).  Each (workgroup, segment) writes one 64x64 fp32
// partial tile; skinny_epilogue_kernel sums a tile's partials in workgroup
// order (deterministic) and applies the same epilogues as the tiled path.
// ---------------------------------------------------------------------------
constexpr int kSkinnyM = 64;      // rows of a skinny pass (decode: one per sequence)
constexpr int kSkinnyBN = 64;     // output columns per tile
constexpr int kSkStages = 4;      // LDS ring depth
constexpr int kSkStage = 2 * 64 * 128;   // A and B, 64 rows x 64 k each: 16 KiB
constexpr int kSkPart = kSkinnyM * kSkinnyBN;   // floats of one partial tile
constexpr int kSkGroups = 512;    // target grid: two workgroups per CU

struct SkSplit {
  int G;        // workgroups
  int U;        // units per workgroup (the last one may hold fewer)
  int KT;       // k steps per tile
  int64_t total;
};

SkSplit skinny_split(int Nt, int K) {
  SkSplit sp;
  sp.KT = K / BK;
  sp.total = (int64_t)(Nt / kSkinnyBN) * sp.KT;
  if (sp.total <= 0) {   // no work (the entry rejects K or N below one tile)
    sp.G = 0;
    sp.U = 1;
    return sp;
  }
  const int64_t g = std::max<int64_t>(1, std::min<int64_t>(kSkGroups, sp.total));
  // at least four k steps (32 KiB of weights) against each 16 KiB partial tile
  sp.U = (int)std::min<int64_t>(std::max<int64_t>((sp.total + g - 1) / g, 4), sp.KT);
  sp.G = (int)((sp.total + sp.U - 1) / sp.U);
  return sp;
}

// Skinny GEMM (M <= 64): workgroup w multiplies the units [w*U, w*U + U) and
// writes the partial tile of each segment to part[w][segment][m][c].  The
// pass streams B (the weights) once, so it is HBM-bound: A and B reach LDS by
// direct loads of whole 128-byte rows (eight lanes per row, one cache line),
// four stages deep, and the four waves each take a 32x32 block of the 64x64
// tile.  The two segments of a range share one load pipeline (the second
// tile's first stages are in flight while the first tile's last ones are
// multiplied); the first segment's accumulators are held in registers and
// both partial tiles are written at the end, so no store sits among the
// loads that the stage waits count.
__global__ __launch_bounds__(256, 2) void gemm_skinny_kernel(GP p, int nb, SkSplit sp,
                                                             float* __restrict__ part) {
  __shared__ __attribute__((aligned(1024))) char sm[kSkStages * kSkStage];
  const int M = p.M_dev ? min(*p.M_dev, p.M_max) : p.M_max;
  if (M <= 0) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t u0 = (int64_t)blockIdx.x * sp.U;
  const int n = (int)(min(sp.total, u0 + sp.U) - u0);   // >= 1: G = ceil(total / U)
  // a range is never longer than a tile's k extent (U <= KT): tiles t0, t1
  const int t0 = (int)(u0 / sp.KT), kb0 = (int)(u0 - (int64_t)t0 * sp.KT);
  const int n0 = min(n, sp.KT - kb0);   // k steps in tile t0; the rest are in t0 + 1
  const int rA = wm * 32 + (lane & 31), rB = wn * 32 + (lane & 31);
  const int swz = (lane >> 1) & 7;
  // direct-load instruction j (0..3) of wave w: operand (A for waves 0-1, B
  // for 2-3), rows 8q .. 8q+7 with q = (4w + j) mod 8; lane l -> row 8q + l/8,
  // stored position l%8, logical chunk (l%8) ^ ((row >> 1) & 7).  src0 / src1
  // point at k step 0 of tile t0 / t0 + 1 (the same A row for both), so the
  // loop only selects one and adds the k offset.
  const bf16* src0[4];
  const bf16* src1[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int q = (4 * wave + j) & 7;
    const int r = 8 * q + (lane >> 3);
    const int ch = (lane & 7) ^ ((r >> 1) & 7);
    if (wave < 2) {
      const int m = min(r, M - 1);   // clamped: loaded, never stored
      const int row = p.a_rows ? p.a_rows[m] : m;
      const bf16* abase = (p.a_sel && (p.a_sel[row] & 1)) ? p.A2 : p.A;
      src0[j] = src1[j] = abase + (int64_t)row * p.lda + ch * 8;
    } else {
      // tile t0 + 1 past the last tile (then n0 == n) is never loaded
      const int na = t0 * kSkinnyBN + r;
      const int nb1 = (int64_t)(t0 + 1) * sp.KT < sp.total ? na + kSkinnyBN : na;
      src0[j] = (na >= nb ? p.B2 + (int64_t)(na - nb) * p.ldb : p.B + (int64_t)na * p.ldb) + ch * 8;
      src1[j] = (nb1 >= nb ? p.B2 + (int64_t)(nb1 - nb) * p.ldb : p.B + (int64_t)nb1 * p.ldb) +
                ch * 8;
    }
  }
  auto issue = [&](int i) {   // stage i of the range into ring slot i % kSkStages
    const bool second = i >= n0;
    const int k = (second ? i - n0 : kb0 + i) * BK;
    char* slot = sm + (i % kSkStages) * kSkStage + (wave >> 1) * 8192;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      dma16((second ? src1[j] : src0[j]) + k, slot + ((4 * wave + j) & 7) * 1024);
  };
  // the stages [i0, i1) of the range into acc
  auto run = [&](f32x16_t& acc, int i0, int i1) {
    for (int it = i0; it < i1; ++it) {
      // stage it has landed once at most the later stages' loads are in
      // flight; near the end of the range fewer stages follow it
      if (it + kSkStages - 2 < n) wait_vm<4 * (kSkStages - 2)>();
      else wait_dma();
      stage_barrier();   // publishes stage it; every wave is done with stage it-1
      if (it + kSkStages - 1 < n) issue(it + kSkStages - 1);   // into stage it-1's slot
      const char* st = sm + (it % kSkStages) * kSkStage;
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = (2 * ks + (lane >> 5)) ^ swz;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(st + (rA * 8 + ch) * 16);
        const bf16x8_t b = *reinterpret_cast<const bf16x8_t*>(st + 8192 + (rB * 8 + ch) * 16);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
      }
    }
  };
  f32x16_t acc0, acc1;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc0[v] = acc1[v] = 0.0f;
#pragma unroll
  for (int s = 0; s < kSkStages - 1; ++s)
    if (s < n) issue(s);
  run(acc0, 0, n0);
  run(acc1, n0, n);
  // every load has landed (the last stage waited for all of them)
  // C layout: value v is row 8*(v/4) + 4*(lane/32) + v%4 of the block, column lane%32
  float* dst = part + (int64_t)blockIdx.x * 2 * kSkPart;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int r = wm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    dst[r * kSkinnyBN + wn * 32 + (lane & 31)] = acc0[v];
  }
  if (n0 < n) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = wm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
      dst[kSkPart + r * kSkinnyBN + wn * 32 + (lane & 31)] = acc1[v];
    }
  }
}

// Sum of the partials of row m, partial-space columns c..c+3: the
// workgroups whose ranges meet c's tile, in ascending order; a workgroup
// whose range starts in that tile holds it as segment 0, one that starts in
// the tile before as segment 1.
__device__ __forceinline__ float4 skinny_sum(const float* __restrict__ part, const SkSplit& sp,
                                             int m, int c) {
  const int t = c / kSkinnyBN, col = c - t * kSkinnyBN;
  const int64_t u0 = (int64_t)t * sp.KT;
  const int w0 = (int)(u0 / sp.U), w1 = (int)((u0 + sp.KT - 1) / sp.U);
  float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int w = w0; w <= w1; ++w) {
    const int seg = (int64_t)w * sp.U >= u0 ? 0 : 1;
    const float4 y = *reinterpret_cast<const float4*>(part + ((int64_t)w * 2 + seg) * kSkPart +
                                                      m * kSkinnyBN + col);
    x.x += y.x; x.y += y.y; x.z += y.z; x.w += y.w;
  }
  return x;
}

// One thread per (row, 4 output columns).
template <int EPI>
__global__ __launch_bounds__(256) void skinny_epilogue_kernel(GP p, int nout, SkSplit sp,
                                                              const float* __restrict__ part) {
  const int M = p.M_dev ? min(*p.M_dev, p.M_max) : p.M_max;
  const int g4 = nout / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int m = (int)(idx / g4), n = (int)(idx % g4) * 4;
  if (m >= M) return;
  const float sc = p.row_scale ? p.row_scale[m] : 1.0f;
  const float4 x4 = skinny_sum(part, sp, m, n);
  const float4 bx = bias4(p.bias, n);
  const float x[4] = {x4.x * sc + bx.x, x4.y * sc + bx.y, x4.z * sc + bx.z, x4.w * sc + bx.w};
  bf16x4_t o;
  if (EPI == EPI_GELU || EPI == EPI_GELU_TANH) {
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = f2bf(EPI == EPI_GELU ? gelu_erf(x[e]) : gelu_tanh(x[e]));
    *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + (int64_t)m * p.ldc + n) = o;
  } else if (EPI == EPI_STORE) {
    const int64_t off = (int64_t)m * p.ldc + n;
    if (p.c_f32) {
      *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.C) + off) =
          make_float4(x[0], x[1], x[2], x[3]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = f2bf(x[e]);
      *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + off) = o;
    }
  } else if (EPI == EPI_RESID) {
    const int64_t off = (int64_t)p.rows[m] * p.ldc + n;
    const bf16x4_t r = *reinterpret_cast<const bf16x4_t*>(p.resid + off);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = f2bf(x[e] + bf2f(r[e]));
    *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + off) = o;
  } else if (EPI == EPI_SWIGLU) {
    const float4 u4 = skinny_sum(part, sp, m, nout + n);
    const float u[4] = {u4.x * sc, u4.y * sc, u4.z * sc, u4.w * sc};
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = f2bf(silu(x[e]) * u[e]);
    *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + (int64_t)m * p.ldc + n) = o;
  } else {  // EPI_QKV
    const int sec = n / p.d_q, cin = n - sec * p.d_q;
    const int row = p.rows[m];
    const bool is_v = sec == 2;
    bf16* dst = sec == 0 ? p.q_out + (int64_t)m * p.d_q
                         : (is_v ? p.v_cache : p.k_cache) +
                               (int64_t)(p.slot ? p.slot[row] : row) * p.d_q;
    if (is_v || !p.rope_cos) {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = f2bf(x[e]);
    } else {
      // rotate-half RoPE: column c pairs with c +- hd/2 of the same head
      const int hd = p.head_dim, half = hd >> 1;
      const int c = cin & (hd - 1);
      const float4 y4 = skinny_sum(part, sp, m, n ^ half);
      const float4 by = bias4(p.bias, n ^ half);
      const float y[4] = {y4.x * sc + by.x, y4.y * sc + by.y, y4.z * sc + by.z, y4.w * sc + by.w};
      const int64_t t = (int64_t)p.pos[row] * half + (c & (half - 1));
      const float4 cs = *reinterpret_cast<const float4*>(p.rope_cos + t);
      const float4 sn = *reinterpret_cast<const float4*>(p.rope_sin + t);
      const float cv[4] = {cs.x, cs.y, cs.z, cs.w}, sv[4] = {sn.x, sn.y, sn.z, sn.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = f2bf(c < half ? x[e] * cv[e] - y[e] * sv[e] : x[e] * cv[e] + y[e] * sv[e]);
    }
    *reinterpret_cast<bf16x4_t*>(dst + cin) = o;
  }
}

// The residual epilogue with the next step over its result rows: one
// workgroup of 1024 threads per row m (rows of at most 4096; thread t owns
// columns 4t..4t+3, so every partial of the row is in flight at once).  From
// the bf16 results (the values a separate pass would read back), summed lane
// by lane, across the wave, then over the 16 waves in order:
//  * ROW_RINV: rinv_out[m] = 1/sqrt(mean(v^2) + eps) (the next RMSNorm's
//    factor), f32;
//  * ROW_LN: ln_out[m] = (v - mean) / sqrt(var + eps) (LayerNorm without its
//    affine part, two passes over the registers), f32;
//  * ROW_EXIT: the GLOBAL exit test of the row against its inertia I:
//    <v,v>, <I,I>, <v,I> in double (every product of two floats is exact),
//    the decision of Eq. 8, then I += v/|v| (as adept_exit_test).
enum { ROW_RINV = 0, ROW_LN = 1, ROW_EXIT = 2 };
template <int MODE>
__global__ __launch_bounds__(1024) void skinny_resid_row_kernel(GP p, int nout, SkSplit sp,
                                                                const float* __restrict__ part) {
  __shared__ float wsum[16];
  __shared__ float total;
  __shared__ double dsum[16][3];
  __shared__ double dtot[3];
  const int M = p.M_dev ? min(*p.M_dev, p.M_max) : p.M_max;
  const int m = blockIdx.x;
  if (m >= M) return;
  const float sc = p.row_scale ? p.row_scale[m] : 1.0f;
  const int n = threadIdx.x * 4;
  const bool live = n < nout;
  float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (live) {
    const float4 x4 = skinny_sum(part, sp, m, n);
    const float4 bx = bias4(p.bias, n);
    const float x[4] = {x4.x * sc + bx.x, x4.y * sc + bx.y, x4.z * sc + bx.z, x4.w * sc + bx.w};
    const int64_t off = (int64_t)p.rows[m] * p.ldc + n;
    const bf16x4_t r = *reinterpret_cast<const bf16x4_t*>(p.resid + off);
    bf16x4_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = f2bf(x[e] + bf2f(r[e]));
      v[e] = bf2f(o[e]);
    }
    *reinterpret_cast<bf16x4_t*>(reinterpret_cast<bf16*>(p.C) + off) = o;
  }
  auto block_sum = [&](float x) {
    x = wave_sum_f32(x);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
      float t = 0.0f;
#pragma unroll
      for (int w = 0; w < 16; ++w) t += wsum[w];
      total = t;
    }
    __syncthreads();
    const float t = total;
    __syncthreads();   // wsum and total are reused by the next sum
    return t;
  };
  if (MODE == ROW_EXIT) {
    const int row = p.rows[m];
    float* ir = p.ex.inertia + (int64_t)row * nout;
    f32x4_t i4 = {0.f, 0.f, 0.f, 0.f};
    if (live) i4 = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(ir + n));
    const float iv[4] = {i4[0], i4[1], i4[2], i4[3]};
    double s3[3] = {0.0, 0.0, 0.0};   // <v,v>, <I,I>, <v,I>
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double a = v[e], b = iv[e];
      s3[0] = fma(a, a, s3[0]);
      s3[1] = fma(b, b, s3[1]);
      s3[2] = fma(a, b, s3[2]);
    }
#pragma unroll
    for (int q = 0; q < 3; ++q) s3[q] = wave_sum_f64(s3[q]);
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
      for (int q = 0; q < 3; ++q) dsum[threadIdx.x >> 6][q] = s3[q];
    }
    __syncthreads();
    if (threadIdx.x < 3) {
      double t = 0.0;
#pragma unroll
      for (int w = 0; w < 16; ++w) t += dsum[w][threadIdx.x];
      dtot[threadIdx.x] = t;
    }
    __syncthreads();
    const double nh = sqrt(dtot[0]), nr = sqrt(dtot[1]);
    const double den = nh * nr;
    const double sim = den > 0.0 ? dtot[2] / den : __longlong_as_double(0x7ff8000000000000ll);
    if (threadIdx.x == 0) {
      p.ex.exit_flag[m] = exit_decision(sim >= p.ex.delta, p.ex.layer, p.ex.min_exit_layer,
                                        p.ex.n_layers, p.ex.force_layer, row) ? 1 : 0;
      if (p.ex.sim_out) p.ex.sim_out[m] = sim;
    }
    if (live && nh > 0.0) {
      const double inv = 1.0 / nh;
      f32x4_t o4;
#pragma unroll
      for (int e = 0; e < 4; ++e) o4[e] = (float)((double)iv[e] + (double)v[e] * inv);
      __builtin_nontemporal_store(o4, reinterpret_cast<f32x4_t*>(ir + n));
    }
  } else if (MODE == ROW_RINV) {
    float ss = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) ss = fmaf(v[e], v[e], ss);
    const float t = block_sum(ss);
    if (threadIdx.x == 0) p.rinv_out[m] = 1.0f / sqrtf(t / (float)nout + p.row_eps);
  } else {
    const float mean = block_sum((v[0] + v[1]) + (v[2] + v[3])) / (float)nout;
    float q = 0.0f;
    if (live) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = v[e] - mean;
        q = fmaf(t, t, q);
      }
    }
    const float r = 1.0f / sqrtf(block_sum(q) / (float)nout + p.row_eps);
    if (live) {
      bf16x4_t y;
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = f2bf((v[e] - mean) * r);
      *reinterpret_cast<bf16x4_t*>(p.ln_out + (int64_t)m * nout + n) = y;
    }
  }
}

template <int EPI>
adept_status launch_skinny(const GP& p, int Nt, int nout, hipStream_t s, const char* name,
                           float* part) {
  const SkSplit sp = skinny_split(Nt, p.K);
  {
    TimedLaunch tl(name ? name : "gemm_skinny", s);
    hipLaunchKernelGGL(gemm_skinny_kernel, dim3(sp.G), dim3(256), 0, s, p,
                       EPI == EPI_SWIGLU ? nout : Nt, sp, part);
  }
  ADEPT_CHECK_LAUNCH("gemm_skinny");
  if (EPI == EPI_RESID && (p.ln_out || p.rinv_out || p.has_exit)) {
    const dim3 g(p.M_max), b(1024);
    if (p.has_exit)
      ADEPT_LAUNCH(skinny_resid_row_kernel<ROW_EXIT>, g, b, 0, s, p, nout, sp, part);
    else if (p.ln_out)
      ADEPT_LAUNCH(skinny_resid_row_kernel<ROW_LN>, g, b, 0, s, p, nout, sp, part);
    else
      ADEPT_LAUNCH(skinny_resid_row_kernel<ROW_RINV>, g, b, 0, s, p, nout, sp, part);
    return launch_status("skinny_resid_row");
  }
  const int64_t total = (int64_t)p.M_max * (nout / 4);
  ADEPT_LAUNCH(skinny_epilogue_kernel<EPI>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
               s, p, nout, sp, part);
  return launch_status("skinny_epilogue");
}

GP to_gp(const GemmArgs& g) {
  GP p{};
  p.M_max = g.M_max; p.M_dev = g.M_dev; p.N = g.N; p.K = g.K;
  p.A = (const bf16*)g.A; p.a_rows = g.a_rows; p.lda = g.lda;
  p.B = (const bf16*)g.B; p.B2 = (const bf16*)g.B2; p.ldb = g.ldb;
  p.C = g.C; p.ldc = g.ldc; p.c_f32 = g.c_f32; p.row_scale = g.row_scale;
  p.rows = g.rows; p.resid = (const bf16*)g.resid; p.pos = g.pos; p.slot = g.slot;
  p.bias = (const bf16*)g.bias;
  p.rope_cos = g.rope_cos; p.rope_sin = g.rope_sin; p.head_dim = g.head_dim; p.d_q = g.d_q;
  p.q_out = (bf16*)g.q_out; p.k_cache = (bf16*)g.k_cache; p.v_cache = (bf16*)g.v_cache;
  p.bias_layer_stride = g.bias_layer_stride; p.a_sorted = g.a_sorted;
  p.A2 = (const bf16*)g.A2; p.a_sel = g.a_sel;
  p.rinv_out = g.rinv_out; p.ln_out = (bf16*)g.ln_out; p.row_eps = g.row_eps;
  p.has_exit = g.exit != nullptr;
  if (g.exit) p.ex = *g.exit;
  return p;
}

bool aligned8(const void* p) { return ((uintptr_t)p & 7u) == 0; }

bool aligned_operands(const GemmArgs& g) {
  return aligned16(g.A) && aligned16(g.B) && (!g.B2 || aligned16(g.B2)) &&
         (!g.a_sel || (g.A2 && aligned16(g.A2))) && g.lda % 8 == 0 &&
         g.ldb % 8 == 0;
}

}  // namespace

size_t skinny_ws_bytes(int Nt, int K) {
  return (size_t)skinny_split(Nt, K).G * 2 * kSkPart * sizeof(float);
}

bool gemm_skinny_row_norm(const GemmArgs& g) {
  return g.epi == EPI_RESID && g.M_max > 0 && g.M_max <= kSkinnyM && g.skinny_ws && g.N > 0 &&
         g.N % 64 == 0 && g.N <= 4096 && g.K > 0 && g.K % BK == 0 &&
         skinny_ws_bytes(g.N, g.K) <= g.skinny_ws_bytes;
}

adept_status gemm(adept_dtype dt, const GemmArgs& g, hipStream_t s) {
  if (g.M_max <= 0) return ADEPT_OK;
  if ((g.rinv_out || g.ln_out || g.exit) &&
      (!gemm_skinny_row_norm(g) || (!!g.rinv_out + !!g.ln_out + !!g.exit) > 1 ||
       (g.ln_out && !aligned8(g.ln_out)) ||
       (g.exit && (!g.exit->inertia || !aligned16(g.exit->inertia) || !g.exit->exit_flag)))) {
    set_error("gemm: one of rinv_out / ln_out (8-byte aligned) / exit (16-byte aligned inertia, "
              "flags) only on the skinny residual path (see gemm_skinny_row_norm)");
    return ADEPT_E_INVALID;
  }
  if (dt != ADEPT_BF16) {
    set_error("gemm: bf16 entry called with another dtype");
    return ADEPT_E_INVALID;
  }
  if (g.K <= 0 || g.K % BK != 0) {
    set_error("gemm: K=%d not a positive multiple of %d", g.K, BK);
    return ADEPT_E_UNSUPPORTED;
  }
  // the last 256-column tile may be ragged (N a multiple of 64); SwiGLU pairs
  // 64 gate with 64 up columns per wave, so its N is a multiple of 128
  const int ncols = g.epi == EPI_SWIGLU ? 128 : 64;
  if (g.N <= 0 || g.N % ncols != 0) {
    set_error("gemm: N=%d not a positive multiple of %d", g.N, ncols);
    return ADEPT_E_UNSUPPORTED;
  }
  if ((g.epi == EPI_QKV) &&
      (g.d_q % 64 != 0 ||
       (g.rope_cos && (g.d_q % 128 != 0 || (g.head_dim != 64 && g.head_dim != 128))) ||
       (!g.rope_cos && !g.bias && g.d_q % 128 != 0))) {
    set_error("gemm: QKV epilogue needs d_q %% 64 == 0 (d_q %% 128 == 0 and head_dim 64/128 "
              "with RoPE or without a bias)");
    return ADEPT_E_UNSUPPORTED;
  }
  if (g.bias && (g.epi == EPI_SWIGLU || g.epi == EPI_KV || !aligned8(g.bias))) {
    set_error("gemm: bias needs an 8-byte aligned [N] vector and no SWIGLU / KV epilogue");
    return ADEPT_E_UNSUPPORTED;
  }
  if (!aligned_operands(g)) {
    set_error("gemm: operands must be 16-byte aligned with leading dims a multiple of 8");
    return ADEPT_E_INVALID;
  }
  GP p = to_gp(g);
  if (g.M_max <= kSkinnyM && g.skinny_ws && g.epi != EPI_KV) {
    const int Nt = g.epi == EPI_SWIGLU ? 2 * g.N : g.N;
    if (skinny_ws_bytes(Nt, g.K) <= g.skinny_ws_bytes) {
      switch (g.epi) {
        case EPI_STORE: return launch_skinny<EPI_STORE>(p, Nt, g.N, s, g.name, g.skinny_ws);
        case EPI_QKV: return launch_skinny<EPI_QKV>(p, Nt, g.N, s, g.name, g.skinny_ws);
        case EPI_RESID: return launch_skinny<EPI_RESID>(p, Nt, g.N, s, g.name, g.skinny_ws);
        case EPI_SWIGLU: return launch_skinny<EPI_SWIGLU>(p, Nt, g.N, s, g.name, g.skinny_ws);
        case EPI_GELU: return launch_skinny<EPI_GELU>(p, Nt, g.N, s, g.name, g.skinny_ws);
        case EPI_GELU_TANH:
          return launch_skinny<EPI_GELU_TANH>(p, Nt, g.N, s, g.name, g.skinny_ws);
        default: break;
      }
    }
  }
  p.tiles_m = ceil_div(g.M_max, BM);
  p.tiles_n = g.epi == EPI_SWIGLU ? g.N / 128 : ceil_div(g.N, BN);
  switch (g.epi) {
    case EPI_STORE: return launch_bf16<EPI_STORE, 0>(p, s, g.name);
    case EPI_QKV:
      return g.head_dim == 128 ? launch_bf16<EPI_QKV, 128>(p, s, g.name)
                               : launch_bf16<EPI_QKV, 64>(p, s, g.name);
    case EPI_RESID: return launch_bf16<EPI_RESID, 0>(p, s, g.name);
    case EPI_SWIGLU: return launch_bf16<EPI_SWIGLU, 0>(p, s, g.name);
    case EPI_GELU: return launch_bf16<EPI_GELU, 0>(p, s, g.name);
    case EPI_GELU_TANH: return launch_bf16<EPI_GELU_TANH, 0>(p, s, g.name);
    default: set_error("gemm: bad epilogue"); return ADEPT_E_INVALID;
  }
}

// f32 GEMM + element-wise epilogue; tmp holds M_max x (N or 2N for SWIGLU) floats.
adept_status gemm_f32(const GemmArgs& g, float* tmp, hipStream_t s) {
  if (g.M_max <= 0) return ADEPT_OK;
  const int nt = g.epi == EPI_SWIGLU ? 2 * g.N : g.N;
  dim3 block(256);
  dim3 grid(ceil_div(g.M_max, FT), ceil_div(g.N, FT));
  ADEPT_LAUNCH(gemm_f32_kernel, grid, block, 0, s, g.M_max, g.M_dev, g.N, g.K,
               (const float*)g.A, g.a_rows, g.lda, (const float*)g.B, g.ldb, tmp, (int64_t)nt);
  ADEPT_CHECK_LAUNCH("gemm_f32");
  if (g.epi == EPI_SWIGLU) {
    ADEPT_LAUNCH(gemm_f32_kernel, grid, block, 0, s, g.M_max, g.M_dev, g.N, g.K,
                 (const float*)g.A, g.a_rows, g.lda, (const float*)g.B2, g.ldb, tmp + g.N,
                 (int64_t)nt);
    ADEPT_CHECK_LAUNCH("gemm_f32");
  }
  GP p = to_gp(g);
  const int64_t total = (int64_t)g.M_max * g.N;
  ADEPT_LAUNCH(epilogue_f32_kernel, dim3((unsigned)((total + 255) / 256)), block, 0, s, g.epi,
               g.M_max, g.M_dev, g.N, (const float*)tmp, (int64_t)nt, p);
  return launch_status("epilogue_f32");
}

// f32 GEMM written straight to C (no epilogue, no row scale): C[m][n] = A[m] . B[n].
adept_status gemm_f32_direct(const GemmArgs& g, hipStream_t s) {
  if (g.M_max <= 0) return ADEPT_OK;
  dim3 grid(ceil_div(g.M_max, FT), ceil_div(g.N, FT));
  ADEPT_LAUNCH(gemm_f32_kernel, grid, dim3(256), 0, s, g.M_max, g.M_dev, g.N, g.K,
               (const float*)g.A, g.a_rows, g.lda, (const float*)g.B, g.ldb, (float*)g.C, g.ldc);
  return launch_status("gemm_f32");
}

// Grouped bf16 GEMM of the KV generation (see the header comment).  g.row_scale
// is indexed by the sorted position.
adept_status gemm_kv_grouped(const GemmArgs& g, const int32_t* work, const int32_t* n_work,
                             int max_work, const int32_t* grp_m,
                             const int32_t* srows,
                             int64_t b_layer_stride, int64_t cache_layer_stride, hipStream_t s) {
  if (max_work <= 0) return ADEPT_OK;
  if (!aligned_operands(g)) {
    set_error("kv_generate: operands must be 16-byte aligned");
    return ADEPT_E_INVALID;
  }
  if (g.N <= 0 || g.N % 64 != 0 || (g.bias && !aligned8(g.bias)) ||
      (!g.bias && g.d_q % 128 != 0)) {
    set_error("kv_generate: 2*H*hd must be a multiple of 64 (128 per section without a bias), "
              "the bias 8-byte aligned");
    return ADEPT_E_UNSUPPORTED;
  }
  GP p = to_gp(g);
  p.work = work; p.n_work = n_work; p.grp_m = grp_m; p.srows = srows;
  p.b_layer_stride = b_layer_stride;
  p.cache_layer_stride = cache_layer_stride;
  p.tiles_n = ceil_div(g.N, BN);
  const bool ext = needs_ext(p, EPI_KV) || (g.bias != nullptr);
  // one workgroup per item: the host bound on the items, rounded to whole XCD rounds
  const int flat = (max_work * p.tiles_n + 7) / 8 * 8;
  if (g.head_dim == 128 && !ext) {
    static bool attr_set = false;
    ADEPT_TRY(allow_lds((const void*)gemm_kv_flat_kernel<128, false>, &attr_set, "kv LDS limit"));
    ADEPT_LAUNCH((gemm_kv_flat_kernel<128, false>), dim3(flat), dim3(kThreads), kLdsBytes, s, p);
  } else if (g.head_dim == 128) {
    static bool attr_set = false;
    ADEPT_TRY(allow_lds((const void*)gemm_kv_flat_kernel<128, true>, &attr_set, "kv LDS limit"));
    ADEPT_LAUNCH((gemm_kv_flat_kernel<128, true>), dim3(flat), dim3(kThreads), kLdsBytes, s, p);
  } else if (!ext) {
    static bool attr_set = false;
    ADEPT_TRY(allow_lds((const void*)gemm_kv_flat_kernel<64, false>, &attr_set, "kv LDS limit"));
    ADEPT_LAUNCH((gemm_kv_flat_kernel<64, false>), dim3(flat), dim3(kThreads), kLdsBytes, s, p);
  } else {
    static bool attr_set = false;
    ADEPT_TRY(allow_lds((const void*)gemm_kv_flat_kernel<64, true>, &attr_set, "kv LDS limit"));
    ADEPT_LAUNCH((gemm_kv_flat_kernel<64, true>), dim3(flat), dim3(kThreads), kLdsBytes, s, p);
  }
  return launch_status("gemm_kv_grouped");
}

}  // namespace adept
