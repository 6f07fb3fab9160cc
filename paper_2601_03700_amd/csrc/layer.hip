// One decoder layer of the generative early-exit forward (Appendix I):
// regular processing of the active rows, then the exit test, the active-list
// update and the KV generation for the rows that exit.  Everything is
// enqueued on one stream with the variable counts kept on the device.
//
// With one query row per sequence (decode) no row of the pass reads another
// row's cache entries, so the K/V a row generates for its skipped layers
// (Eq. 9) are needed only by later passes.  Two schedules use that:
//  * deferred: the generation of all rows runs after layer N, as one grouped
//    GEMM in which each skipped layer's Wk/Wv is read once;
//  * fused (kv_fused): layer r's QKV GEMM also takes the rows that exited
//    before r, reading their exit state, so their K/V at layer r come out of
//    the GEMM that reads layer r's weights anyway (Eq. 6 leaves the order of
//    the generation free); the Q columns of those rows are computed and
//    ignored.  In a decode pass the GEMM streams its weights once whatever
//    its row count, so the generation costs no weight traffic.
#include <algorithm>

#include "common.h"

namespace adept {
namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct LayerWs {
  float* rinv;    // [n_tok] 1/rms of the active rows (compact order)
  void* compact;  size_t compact_bytes;
  void* attend;   size_t attend_bytes;
  void* kvgen;    size_t kvgen_bytes;
  int32_t* all_rows;  // [n_tok + 64]: row list and its count (deferred / fused KV generation)
  int32_t* fsel;      // [n_tok]: fused schedule, 1 where a row's exit state is in h[layer & 1]
  void* prompt;   size_t prompt_bytes;   // per-sequence keys of the all-at-once variant
  void* hsm;      size_t hsm_bytes;      // mapper activations (when a mapper is given)
  float* skinny;  size_t skinny_bytes;   // GEMM partial sums when n_tok <= 64 (decode)
  float* gemm_tmp;  // f32 path only
  void* xnorm;      // [n_tok][D] normalised rows (GPT2 family)
  size_t total;
};

LayerWs carve(const adept_layer_args* a, void* base) {
  LayerWs w{};
  char* p = (char*)base;
  size_t off = 0;
  const int dq = a->n_heads * a->head_dim;
  w.rinv = (float*)(p + off); off += align256((size_t)a->n_tok * sizeof(float));
  w.compact_bytes = adept_compact_workspace_bytes(a->n_tok);
  w.compact = p + off; off += align256(w.compact_bytes);
  w.attend_bytes = attend_workspace_bytes(a->n_tok, a->n_seq, a->n_heads, a->head_dim, a->s_max);
  w.attend = p + off; off += align256(w.attend_bytes);
  const bool gpt2 = a->family == ADEPT_FAMILY_GPT2;
  w.kvgen_bytes = gpt2 ? adept_kv_generate_layernorm_workspace_bytes(a->n_layers, a->n_tok,
                                                                     a->d_model)
                       : adept_kv_generate_workspace_bytes(a->n_layers, a->n_tok);
  w.kvgen = p + off; off += align256(w.kvgen_bytes);
  if (gpt2) {
    w.xnorm = p + off;
    off += align256((size_t)a->n_tok * a->d_model * 2);
  }
  w.all_rows = (int32_t*)(p + off); off += align256(((size_t)a->n_tok + 64) * sizeof(int32_t));
  w.fsel = (int32_t*)(p + off); off += align256((size_t)a->n_tok * sizeof(int32_t));
  w.prompt_bytes = adept_exit_prompt_level_workspace_bytes(a->n_seq);
  w.prompt = p + off; off += align256(w.prompt_bytes);
  w.hsm_bytes = a->hsm ? adept_hsm_workspace_bytes(a->d_model, a->n_tok) : 0;
  w.hsm = p + off; off += align256(w.hsm_bytes);
  if (a->dtype == ADEPT_BF16 && a->n_tok <= 64) {
    w.skinny_bytes = std::max({skinny_ws_bytes(3 * dq, a->d_model), skinny_ws_bytes(a->d_model, dq),
                               skinny_ws_bytes(2 * a->d_ff, a->d_model),
                               skinny_ws_bytes(a->d_model, a->d_ff)});
    w.skinny = (float*)(p + off);
    off += align256(w.skinny_bytes);
  }
  if (a->dtype == ADEPT_F32) {
    const size_t cols = std::max({(size_t)3 * dq, (size_t)2 * a->d_ff, (size_t)a->d_model});
    w.gemm_tmp = (float*)(p + off);
    off += align256((size_t)a->n_tok * cols * sizeof(float));
  }
  w.total = off;
  return w;
}

// Deferred KV generation, step 1: the row list 0..n_tok-1 with its count,
// and the exit state of every row that exited at a layer of the other
// parity than N copied into h[N & 1] (one wave per row, 16-byte copies; no
// later kernel reads an exited row of that buffer, and the final head reads
// the same values).
__global__ __launch_bounds__(64) void defer_rows_kernel(int n_tok, int n_layers, int row_bytes,
                                                        const int32_t* __restrict__ exit_layer,
                                                        const char* __restrict__ h_other,
                                                        char* __restrict__ h_last,
                                                        int32_t* __restrict__ rows,
                                                        int32_t* __restrict__ count) {
  const int j = blockIdx.x;
  if (threadIdx.x == 0) {
    rows[j] = j;
    if (j == 0) *count = n_tok;
  }
  const int e = exit_layer[j];
  if (e >= n_layers || ((e ^ n_layers) & 1) == 0) return;
  const int64_t base = (int64_t)j * row_bytes;
  for (int o = threadIdx.x * 16; o < row_bytes; o += 64 * 16)
    *reinterpret_cast<uint4*>(h_last + base + o) = *reinterpret_cast<const uint4*>(h_other + base + o);
}

// Fused schedule, the row list of layer `layer`'s QKV GEMM: the active rows
// (as listed) followed by the rows that exited at a layer below `layer`
// (ascending), and its count; sel[row] = 1 where the row's state (its exit
// state) sits in h[layer & 1] rather than h[(layer-1) & 1].  Written by one
// workgroup; wave 0 walks the rows 64 at a time with a ballot.
__device__ __forceinline__ void fused_rows_write(int n_tok, int layer, int na,
                                                 const int32_t* __restrict__ exit_layer,
                                                 const int32_t* __restrict__ act,
                                                 int32_t* __restrict__ list,
                                                 int32_t* __restrict__ count,
                                                 int32_t* __restrict__ sel) {
  for (int k = threadIdx.x; k < na; k += blockDim.x) list[k] = act[k];
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  const int par = (layer - 1) & 1;
  int off = 0;
  for (int base = 0; base < n_tok; base += 64) {
    const int row = base + lane;
    const int el = row < n_tok ? exit_layer[row] : INT_MAX;
    const bool ex = el < layer;
    const uint64_t m = __ballot(ex);
    if (ex) list[na + off + __popcll(m & ((1ull << lane) - 1))] = row;
    if (row < n_tok) sel[row] = ex && (el & 1) != par;
    off += __popcll(m);
  }
  if (lane == 0) *count = na + off;
}

// Entry k of that list, found by one wave from the same ballots (-1 past its
// end), and whether the row's state is in h[layer & 1].
__device__ __forceinline__ int fused_row_of(int k, int n_tok, int layer, int na,
                                            const int32_t* __restrict__ exit_layer,
                                            const int32_t* __restrict__ act, bool* from_out) {
  const int lane = threadIdx.x & 63;
  *from_out = false;
  if (k < na) return act[k];
  const int want = k - na;   // the want-th row that exited before this layer
  int off = 0;
  for (int base = 0; base < n_tok; base += 64) {
    const int r = base + lane;
    const bool ex = r < n_tok && exit_layer[r] < layer;
    const uint64_t m = __ballot(ex);
    const int c = __popcll(m);
    if (want < off + c) {
      const uint64_t hit = __ballot(ex && __popcll(m & ((1ull << lane) - 1)) == want - off);
      const int row = base + __ffsll((unsigned long long)hit) - 1;
      *from_out = (exit_layer[row] & 1) != ((layer - 1) & 1);
      return row;
    }
    off += c;
  }
  return -1;
}

__global__ __launch_bounds__(256) void fused_rows_kernel(int n_tok, int layer,
                                                         const int32_t* __restrict__ exit_layer,
                                                         const int32_t* __restrict__ act,
                                                         const int32_t* __restrict__ n_act,
                                                         int max_act, int32_t* __restrict__ list,
                                                         int32_t* __restrict__ count,
                                                         int32_t* __restrict__ sel) {
  fused_rows_write(n_tok, layer, min(*n_act, max_act), exit_layer, act, list, count, sel);
}

// The list and the QKV GEMM's row factors in one launch (RMSNorm family):
// workgroup 0 writes the list, every wave finds its own entry k and writes
// rinv[k] = 1/rms of that row's state, so no workgroup waits for another.
// A kernel boundary costs more than the few ballots each wave repeats.
template <typename T>
__global__ __launch_bounds__(256) void fused_rows_rinv_kernel(
    int n_tok, int layer, int d, float eps, const int32_t* __restrict__ exit_layer,
    const int32_t* __restrict__ act, const int32_t* __restrict__ n_act, int max_act,
    const T* __restrict__ x_in, const T* __restrict__ x_out, int32_t* __restrict__ list,
    int32_t* __restrict__ count, int32_t* __restrict__ sel, float* __restrict__ rinv) {
  const int na = min(*n_act, max_act);
  if (blockIdx.x == 0) fused_rows_write(n_tok, layer, na, exit_layer, act, list, count, sel);
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  bool from_out;
  const int row = fused_row_of(k, n_tok, layer, na, exit_layer, act, &from_out);
  if (row < 0) return;   // past the list
  const int lane = threadIdx.x & 63;
  const float r = row_rinv_wave((from_out ? x_out : x_in) + (int64_t)row * d, d, eps, lane);
  if (lane == 0) rinv[k] = r;
}

// The same for the LayerNorm family: each wave writes the normalised row k
// (no affine part: folded into the projection) into xnorm[k].
template <int R>
__global__ __launch_bounds__(256) void fused_rows_ln_kernel(
    int n_tok, int layer, int d, float eps, const int32_t* __restrict__ exit_layer,
    const int32_t* __restrict__ act, const int32_t* __restrict__ n_act, int max_act,
    const bf16* __restrict__ x_in, const bf16* __restrict__ x_out, int32_t* __restrict__ list,
    int32_t* __restrict__ count, int32_t* __restrict__ sel, bf16* __restrict__ xnorm) {
  const int na = min(*n_act, max_act);
  if (blockIdx.x == 0) fused_rows_write(n_tok, layer, na, exit_layer, act, list, count, sel);
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  bool from_out;
  const int row = fused_row_of(k, n_tok, layer, na, exit_layer, act, &from_out);
  if (row < 0) return;
  layernorm_row_vec<R>((from_out ? x_out : x_in) + (int64_t)row * d, d, eps, nullptr, nullptr,
                       xnorm + (int64_t)k * d, threadIdx.x & 63);
}

adept_status run_gemm(adept_dtype dt, const GemmArgs& g, float* tmp, hipStream_t s) {
  return dt == ADEPT_BF16 ? gemm(dt, g, s) : gemm_f32(g, tmp, s);
}

// Eq. 9 for the rows listed in rows / n_rows: the K and V rows of each
// layer's stacked QKV weight (and, for the GPT2 family, of its folded bias).
adept_status kv_generate_family(const adept_layer_args* a, adept_dtype dt, const void* s_map,
                                const int32_t* rows, const int32_t* n_rows, int max_rows,
                                const LayerWs& ws, void* stream) {
  const int N = a->n_layers, D = a->d_model, H = a->n_heads, hd = a->head_dim;
  const int64_t dq = (int64_t)H * hd;
  const size_t esz = dt == ADEPT_BF16 ? 2 : 4;
  const void* wkv = (const char*)a->w_qkv + dq * D * (int64_t)esz;
  if (a->family == ADEPT_FAMILY_GPT2)
    return adept_kv_generate_layernorm(dt, N, D, H, hd, a->rms_eps, s_map, rows, n_rows, max_rows,
                                       a->exit_layer, a->slot, wkv, 3 * dq * D,
                                       (const char*)a->b_qkv + dq * (int64_t)esz, 3 * dq,
                                       a->k_cache, a->v_cache, a->n_slots, ws.kvgen,
                                       ws.kvgen_bytes, stream);
  return adept_kv_generate(dt, N, D, H, hd, a->rms_eps, s_map, rows, n_rows, max_rows,
                           a->exit_layer, a->slot, a->pos, wkv, 3 * dq * D, nullptr, a->rope_cos,
                           a->rope_sin, a->rope_max_pos, a->k_cache, a->v_cache, a->n_slots,
                           ws.kvgen, ws.kvgen_bytes, stream);
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_layer_workspace_bytes(const adept_layer_args* a) {
  if (!a) return 0;
  return carve(a, nullptr).total;
}

extern "C" adept_status adept_layer_step(const adept_layer_args* a, int layer, void* stream) {
  ADEPT_REQUIRE(a != nullptr, "layer_step: args is NULL");
  const adept_dtype dt = (adept_dtype)a->dtype;
  ADEPT_REQUIRE(dt == ADEPT_F32 || dt == ADEPT_BF16, "layer_step: bad dtype");
  const int N = a->n_layers, D = a->d_model, H = a->n_heads, hd = a->head_dim, F = a->d_ff;
  ADEPT_REQUIRE(N >= 1 && layer >= 1 && layer <= N, "layer_step: layer %d outside 1..%d", layer, N);
  ADEPT_REQUIRE(a->exit.n_layers == N, "layer_step: exit.n_layers != n_layers");
  ADEPT_REQUIRE(D > 0 && H > 0 && hd > 0 && F > 0 && a->n_tok > 0, "layer_step: bad sizes");
  ADEPT_REQUIRE(a->max_active >= 0 && a->max_active <= a->n_tok, "layer_step: bad max_active");
  ADEPT_REQUIRE(a->n_seq > 0 && a->s_max > 0 && a->n_slots >= (int64_t)a->n_seq * a->s_max,
                "layer_step: cache smaller than n_seq * s_max");
  const bool gpt2 = a->family == ADEPT_FAMILY_GPT2;
  ADEPT_REQUIRE(a->family == ADEPT_FAMILY_LLAMA || gpt2, "layer_step: bad family %d", a->family);
  ADEPT_REQUIRE(!gpt2 || (dt == ADEPT_BF16 && a->b_qkv && a->b_o && a->b_fc && a->b_proj &&
                          D % 64 == 0 && (H * hd) % 64 == 0 && F % 64 == 0 && !a->hsm),
                "layer_step: the GPT2 family needs bf16, the four biases, no mapper and "
                "d_model, H*hd, d_ff multiples of 64");
  ADEPT_REQUIRE(a->w_qkv && a->w_o && a->w_gate && (gpt2 || a->w_up) && a->w_down &&
                    (gpt2 || (a->rope_cos && a->rope_sin)) && a->h[0] && a->h[1] && a->pos &&
                    a->seq && a->slot &&
                    a->active[0] && a->active[1] && a->n_active[0] && a->n_active[1] &&
                    a->exited && a->n_exited && a->exit_layer && a->exit_flag && a->k_cache &&
                    a->v_cache && a->q_buf && a->attn_out && a->ffn_act,
                "layer_step: NULL pointer in args");
  ADEPT_REQUIRE(!a->kv_fused || (dt == ADEPT_BF16 && a->attn_tiles == 0),
                "layer_step: kv_fused needs bf16 and a decode pass (attn_tiles = 0)");
  ADEPT_REQUIRE(a->exit.metric == ADEPT_SIM_LOCAL || a->inertia,
                "layer_step: GLOBAL/BOTH metrics need inertia");
  ADEPT_REQUIRE(!a->hsm || (dt == ADEPT_BF16 && a->exit.metric != ADEPT_SIM_LOCAL && a->inertia),
                "layer_step: the mapper needs bf16 and the inertia (GLOBAL or BOTH metric)");
  const size_t need = adept_layer_workspace_bytes(a);
  if (!a->workspace || a->workspace_bytes < need) {
    set_error("layer_step: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  LayerWs ws = carve(a, a->workspace);
  hipStream_t s = as_stream(stream);
  const int in = (layer - 1) & 1, out = layer & 1;
  const int32_t* act = a->active[in];
  const int32_t* nact = a->n_active[in];
  const int maxn = a->max_active;
  const int dq = H * hd;
  const size_t esz = dt == ADEPT_BF16 ? 2 : 4;
  auto off = [&](const void* base, int64_t elems) {
    return (const void*)((const char*)base + elems * (int64_t)esz);
  };
  const int64_t li = layer - 1;
  const void* wqkv = off(a->w_qkv, li * 3 * dq * D);
  const void* wo = off(a->w_o, li * (int64_t)D * dq);
  const void* wg = off(a->w_gate, li * (int64_t)F * D);
  const void* wu = a->w_up ? off(a->w_up, li * (int64_t)F * D) : nullptr;
  const void* wd = off(a->w_down, li * (int64_t)D * F);
  void* kc = (void*)off(a->k_cache, li * a->n_slots * dq);
  void* vc = (void*)off(a->v_cache, li * a->n_slots * dq);

  // fused schedule: the QKV GEMM's rows are the active rows, then the rows
  // that exited earlier in the pass (their K/V at this layer, Eq. 9)
  const bool fused = a->kv_fused != 0;
  const int32_t* qrows = act;         // rows of the QKV GEMM
  const int32_t* nq = nact;
  const int qmax = fused ? a->n_tok : maxn;
  // fused schedule: the row list and the QKV rows' norm (the RMSNorm
  // factors, or the LayerNorm rows when they fit one wave's registers) come
  // from one kernel
  const bool rinv_fused = fused && !gpt2 && dt == ADEPT_BF16 && qmax > 0;
  const int ln_r = ceil_div(ceil_div(D, 8), 64);   // 16-byte chunks per lane
  const bool ln_fused = fused && gpt2 && dt == ADEPT_BF16 && qmax > 0 && D % 8 == 0 &&
                        ln_r <= 8 && aligned16(a->h[0]) && aligned16(a->h[1]) &&
                        aligned16(ws.xnorm);
  const dim3 fgrid(ceil_div(std::max(qmax, 1), 4));
  // the GLOBAL exit test (step 8) can run in the down projection's epilogue
  // on the skinny path (each result row tested as it is formed)
  RowExit rx{a->exit.delta, layer, a->exit.min_exit_layer, a->exit.n_layers, a->inertia,
             a->force_layer, a->exit_flag, a->sim_out};
  bool exit_done = false;
  auto exit_in_epilogue = [&](GemmArgs& g) -> adept_status {
    if (dt != ADEPT_BF16 || a->exit.metric != ADEPT_SIM_GLOBAL || !gemm_skinny_row_norm(g))
      return ADEPT_OK;
    // the exit test's argument checks, with no rows to test
    ADEPT_TRY(adept_exit_test(dt, D, layer, &a->exit, act, nact, 0, a->h[out], a->h[in],
                              a->inertia, a->force_layer, a->exit_flag, a->sim_out, stream));
    g.exit = &rx;
    exit_done = true;
    return ADEPT_OK;
  };
  if (rinv_fused) {
    ADEPT_LAUNCH(fused_rows_rinv_kernel<bf16>, fgrid, dim3(256), 0, s, a->n_tok, layer, D,
                 a->rms_eps, a->exit_layer, act, nact, maxn, (const bf16*)a->h[in],
                 (const bf16*)a->h[out], ws.all_rows, ws.all_rows + a->n_tok, ws.fsel, ws.rinv);
    ADEPT_CHECK_LAUNCH("fused_rows_rinv");
  } else if (ln_fused) {
    const bf16 *xi = (const bf16*)a->h[in], *xo = (const bf16*)a->h[out];
    int32_t *lst = ws.all_rows, *cnt = ws.all_rows + a->n_tok;
    bf16* xn = (bf16*)ws.xnorm;
    if (ln_r <= 1)
      ADEPT_LAUNCH(fused_rows_ln_kernel<1>, fgrid, dim3(256), 0, s, a->n_tok, layer, D,
                   a->rms_eps, a->exit_layer, act, nact, maxn, xi, xo, lst, cnt, ws.fsel, xn);
    else if (ln_r <= 2)
      ADEPT_LAUNCH(fused_rows_ln_kernel<2>, fgrid, dim3(256), 0, s, a->n_tok, layer, D,
                   a->rms_eps, a->exit_layer, act, nact, maxn, xi, xo, lst, cnt, ws.fsel, xn);
    else if (ln_r <= 4)
      ADEPT_LAUNCH(fused_rows_ln_kernel<4>, fgrid, dim3(256), 0, s, a->n_tok, layer, D,
                   a->rms_eps, a->exit_layer, act, nact, maxn, xi, xo, lst, cnt, ws.fsel, xn);
    else
      ADEPT_LAUNCH(fused_rows_ln_kernel<8>, fgrid, dim3(256), 0, s, a->n_tok, layer, D,
                   a->rms_eps, a->exit_layer, act, nact, maxn, xi, xo, lst, cnt, ws.fsel, xn);
    ADEPT_CHECK_LAUNCH("fused_rows_ln");
  } else if (fused) {
    ADEPT_LAUNCH(fused_rows_kernel, dim3(1), dim3(256), 0, s, a->n_tok, layer, a->exit_layer, act,
                 nact, maxn, ws.all_rows, ws.all_rows + a->n_tok, ws.fsel);
    ADEPT_CHECK_LAUNCH("fused_rows");
  }
  if (fused) {
    qrows = ws.all_rows;
    nq = ws.all_rows + a->n_tok;
  }
  if (qmax > 0 && gpt2) {
    // LayerNorm family: norms without their affine part (folded into the
    // weights and biases), biased projections, tanh GELU, no RoPE
    const void* bqkv = off(a->b_qkv, li * 3 * dq);
    // 1. LN1 of the QKV rows (compact order; an exited row from its exit state)
    if (!ln_fused)
      ADEPT_TRY(layernorm_rows_sel(dt, D, a->rms_eps, a->h[in], a->h[out],
                                   fused ? ws.fsel : nullptr, qrows, nq, qmax, nullptr, nullptr,
                                   ws.xnorm, s));
    // 2. Q/K/V with bias, own K/V into cache[layer]
    GemmArgs g{};
    g.M_max = qmax; g.M_dev = nq; g.N = 3 * dq; g.K = D;
    g.A = ws.xnorm; g.lda = D; g.B = wqkv; g.ldb = D; g.epi = EPI_QKV; g.bias = bqkv;
    g.rows = qrows; g.pos = a->pos; g.slot = a->slot; g.head_dim = hd; g.d_q = dq;
    g.q_out = a->q_buf; g.k_cache = kc; g.v_cache = vc; g.name = "gemm_qkv";
    g.skinny_ws = ws.skinny; g.skinny_ws_bytes = ws.skinny_bytes;
    ADEPT_TRY(gemm(dt, g, s));
    // 3. attention over the mixed cache
    ADEPT_TRY(attend_dispatch(dt, H, hd, 1.0f / sqrtf((float)hd), 1, a->q_buf, act, nact, maxn,
                              a->pos, a->seq, a->n_seq, kc, vc, a->s_max, nullptr, nullptr,
                              a->attn_out, ws.attend, ws.attend_bytes, a->attn_tiles != 0, s));
    // 4. output projection + bias + residual: h[out] = h[in] + o Wo^T + bo
    GemmArgs go{};
    go.M_max = maxn; go.M_dev = nact; go.N = D; go.K = dq;
    go.A = a->attn_out; go.lda = dq; go.B = wo; go.ldb = dq; go.epi = EPI_RESID;
    go.bias = off(a->b_o, li * D);
    go.C = a->h[out]; go.ldc = D; go.resid = a->h[in]; go.rows = act; go.name = "gemm_o";
    go.skinny_ws = ws.skinny; go.skinny_ws_bytes = ws.skinny_bytes;
    // 5. LN2: on the skinny path the projection's epilogue writes it
    if (gemm_skinny_row_norm(go)) {
      go.ln_out = ws.xnorm;
      go.row_eps = a->rms_eps;
    }
    ADEPT_TRY(gemm(dt, go, s));
    if (!go.ln_out)
      ADEPT_TRY(layernorm_rows_sel(dt, D, a->rms_eps, a->h[out], a->h[out], nullptr, act, nact,
                                   maxn, nullptr, nullptr, ws.xnorm, s));
    // 6. first MLP projection + bias + tanh GELU
    GemmArgs gf{};
    gf.M_max = maxn; gf.M_dev = nact; gf.N = F; gf.K = D;
    gf.A = ws.xnorm; gf.lda = D; gf.B = wg; gf.ldb = D; gf.epi = EPI_GELU_TANH;
    gf.bias = off(a->b_fc, li * F);
    gf.C = a->ffn_act; gf.ldc = F; gf.name = "gemm_fc";
    gf.skinny_ws = ws.skinny; gf.skinny_ws_bytes = ws.skinny_bytes;
    ADEPT_TRY(gemm(dt, gf, s));
    // 7. second MLP projection + bias + residual (in place on h[out])
    GemmArgs gd{};
    gd.M_max = maxn; gd.M_dev = nact; gd.N = D; gd.K = F;
    gd.A = a->ffn_act; gd.lda = F; gd.B = wd; gd.ldb = F; gd.epi = EPI_RESID;
    gd.bias = off(a->b_proj, li * D);
    gd.C = a->h[out]; gd.ldc = D; gd.resid = a->h[out]; gd.rows = act; gd.name = "gemm_proj";
    gd.skinny_ws = ws.skinny; gd.skinny_ws_bytes = ws.skinny_bytes;
    ADEPT_TRY(exit_in_epilogue(gd));
    ADEPT_TRY(gemm(dt, gd, s));
  } else if (qmax > 0) {
    // 1. pre-attention RMSNorm: the gain is folded into W_qkv, the row factor
    //    1/rms(h) scales the GEMM accumulators
    if (!rinv_fused)
      ADEPT_TRY(row_rinv_sel(dt, D, a->rms_eps, a->h[in], a->h[out], fused ? ws.fsel : nullptr,
                             qrows, nq, qmax, ws.rinv, s));
    // 2. Q/K/V projections of the gathered rows, RoPE, own K/V into cache[layer]
    GemmArgs g{};
    g.M_max = qmax; g.M_dev = nq; g.N = 3 * dq; g.K = D;
    g.A = a->h[in]; g.a_rows = qrows; g.lda = D; g.B = wqkv; g.ldb = D; g.epi = EPI_QKV;
    if (fused) { g.A2 = a->h[out]; g.a_sel = ws.fsel; }
    g.row_scale = ws.rinv;
    g.rows = qrows; g.pos = a->pos; g.slot = a->slot;
    g.rope_cos = a->rope_cos; g.rope_sin = a->rope_sin; g.head_dim = hd; g.d_q = dq;
    g.q_out = a->q_buf; g.k_cache = kc; g.v_cache = vc; g.name = "gemm_qkv";
    g.skinny_ws = ws.skinny; g.skinny_ws_bytes = ws.skinny_bytes;
    ADEPT_TRY(run_gemm(dt, g, ws.gemm_tmp, s));
    // 3. attention over the mixed cache
    ADEPT_TRY(attend_dispatch(dt, H, hd, 1.0f / sqrtf((float)hd), 1, a->q_buf, act, nact, maxn,
                              a->pos, a->seq, a->n_seq, kc, vc, a->s_max, nullptr, nullptr,
                              a->attn_out, ws.attend, ws.attend_bytes, a->attn_tiles != 0, s));
    // 4. output projection + residual: h[out] = h[in] + o Wo^T
    GemmArgs go{};
    go.M_max = maxn; go.M_dev = nact; go.N = D; go.K = dq;
    go.A = a->attn_out; go.lda = dq; go.B = wo; go.ldb = dq; go.epi = EPI_RESID;
    go.C = a->h[out]; go.ldc = D; go.resid = a->h[in]; go.rows = act; go.name = "gemm_o";
    go.skinny_ws = ws.skinny; go.skinny_ws_bytes = ws.skinny_bytes;
    // 5. pre-FFN RMSNorm (gain folded into W_gate / W_up): its row factors
    //    come from the projection's epilogue on the skinny path
    if (dt == ADEPT_BF16 && gemm_skinny_row_norm(go)) {
      go.rinv_out = ws.rinv;
      go.row_eps = a->rms_eps;
    }
    ADEPT_TRY(run_gemm(dt, go, ws.gemm_tmp, s));
    if (!go.rinv_out) ADEPT_TRY(row_rinv(dt, D, a->rms_eps, a->h[out], act, nact, maxn, ws.rinv, s));
    // 6. gate/up projections with SwiGLU
    GemmArgs gu{};
    gu.M_max = maxn; gu.M_dev = nact; gu.N = F; gu.K = D;
    gu.A = a->h[out]; gu.a_rows = act; gu.lda = D; gu.B = wg; gu.B2 = wu; gu.ldb = D;
    gu.epi = EPI_SWIGLU; gu.row_scale = ws.rinv;
    gu.C = a->ffn_act; gu.ldc = F; gu.name = "gemm_gate_up";
    gu.skinny_ws = ws.skinny; gu.skinny_ws_bytes = ws.skinny_bytes;
    ADEPT_TRY(run_gemm(dt, gu, ws.gemm_tmp, s));
    // 7. down projection + residual (in place on h[out])
    GemmArgs gd{};
    gd.M_max = maxn; gd.M_dev = nact; gd.N = D; gd.K = F;
    gd.A = a->ffn_act; gd.lda = F; gd.B = wd; gd.ldb = F; gd.epi = EPI_RESID;
    gd.C = a->h[out]; gd.ldc = D; gd.resid = a->h[out]; gd.rows = act; gd.name = "gemm_down";
    gd.skinny_ws = ws.skinny; gd.skinny_ws_bytes = ws.skinny_bytes;
    ADEPT_TRY(exit_in_epilogue(gd));
    ADEPT_TRY(run_gemm(dt, gd, ws.gemm_tmp, s));
  }
  // 8. exit test (Eq. 7-8), unless the down projection's epilogue ran it
  if (!exit_done)
    ADEPT_TRY(adept_exit_test(dt, D, layer, &a->exit, act, nact, maxn, a->h[out], a->h[in],
                              a->inertia, a->force_layer, a->exit_flag, a->sim_out, stream));
  // all-at-once variant (Appendix H.2): a prompt's last token decides for all of it
  if (a->exit.prompt_level && a->attn_tiles)
    ADEPT_TRY(adept_exit_prompt_level(act, nact, maxn, a->seq, a->pos, a->n_seq, a->exit_flag,
                                      ws.prompt, ws.prompt_bytes, stream));
  // 9. active-list update
  ADEPT_TRY(adept_compact(layer, N, a->exit_flag, act, nact, maxn, a->active[out], a->n_active[out],
                          a->exited, a->n_exited, a->exit_layer, ws.compact, ws.compact_bytes,
                          stream));
  // 9b. mapper (Section 4.2) of the rows that exited here: s~ replaces h_i
  //     in place, so the K/V generation and the final state use it
  if (a->hsm && layer < N && maxn > 0)
    ADEPT_TRY(adept_hsm_forward(dt, D, a->rms_eps, a->hsm, a->exited, a->n_exited, maxn,
                                a->h[out], a->h[in], a->inertia, 1, a->h[out], ws.hsm,
                                ws.hsm_bytes, stream));
  // 10. K/V of the skipped layers of the rows that exited here (Eq. 9); in
  //     decode, of every row that exited in the pass, after layer N
  const bool defer = a->attn_tiles == 0;
  if (defer && !fused && layer == N) {
    const int rb = D * (dt == ADEPT_BF16 ? 2 : 4);
    ADEPT_LAUNCH(defer_rows_kernel, dim3(a->n_tok), dim3(64), 0, s, a->n_tok, N, rb,
                 a->exit_layer, (const char*)a->h[(N + 1) & 1], (char*)a->h[N & 1], ws.all_rows,
                 ws.all_rows + a->n_tok);
    ADEPT_CHECK_LAUNCH("defer_rows");
    ADEPT_TRY(kv_generate_family(a, dt, a->h[N & 1], ws.all_rows, ws.all_rows + a->n_tok,
                                 a->n_tok, ws, stream));
  }
  if (!defer && layer < N && maxn > 0) {
    ADEPT_TRY(kv_generate_family(a, dt, a->h[out], a->exited, a->n_exited, maxn, ws, stream));
  }
  return ADEPT_OK;
}
