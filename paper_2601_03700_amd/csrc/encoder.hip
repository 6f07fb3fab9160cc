// Classification mode of the token-level exit (Section 4.3, downstream
// tasks): a post-norm encoder (BERT-style) whose tokens stop at their exit
// layer and leave the key set of every later layer; there is no KV
// generation.  A sequence's output is its first ([CLS]) row at that row's
// exit, fed to a linear head.
//
// Layer i on the active rows (all of it enqueued on one stream, counts on the
// device): QKV GEMM + bias (K/V of the row at its own slot) -> bidirectional
// attention over the live rows of the sequence -> O GEMM + bias + residual ->
// LayerNorm -> GEMM + bias + GELU -> GEMM + bias + residual -> LayerNorm ->
// exit test -> active-list update -> the exited rows' keys marked dead.  The
// residual stream ping-pongs between h[0] and h[1] as in the decoder, so an
// exited row keeps its state at exit in h[exit_layer & 1].
#include <algorithm>

#include "common.h"

namespace adept {
namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// One wave per row k < min(*n_dev, max_n): out[row] = LN(x[row]) * g + b
// (row = rows ? rows[k] : k; f32 statistics, two passes; in place allowed).
__global__ __launch_bounds__(256) void layernorm_kernel(int d, float eps,
                                                        const bf16* x,
                                                        const int32_t* __restrict__ rows,
                                                        const int32_t* __restrict__ n_dev,
                                                        int max_n, const bf16* __restrict__ g,
                                                        const bf16* __restrict__ b, bf16* out) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(*n_dev, max_n) : max_n;
  if (k >= n) return;
  const int64_t row = rows ? rows[k] : k;
  const bf16* xr = x + row * d;
  float s = 0.0f;
  for (int c = lane; c < d; c += 64) s += bf2f(xr[c]);
  const float mean = wave_sum_f32(s) / (float)d;
  float v = 0.0f;
  for (int c = lane; c < d; c += 64) {
    const float t = bf2f(xr[c]) - mean;
    v = fmaf(t, t, v);
  }
  const float r = 1.0f / sqrtf(wave_sum_f32(v) / (float)d + eps);
  bf16* o = out + row * d;
  for (int c = lane; c < d; c += 64) o[c] = f2bf((bf2f(xr[c]) - mean) * r * bf2f(g[c]) + bf2f(b[c]));
}

// One wave per row: h0 = LN(word[id] + pos_emb[pos] + type_emb).
__global__ __launch_bounds__(256) void encoder_embed_kernel(
    int n, int d, int vocab, int max_pos, float eps, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ pos, const bf16* __restrict__ word, const bf16* __restrict__ pemb,
    const bf16* __restrict__ temb, const bf16* __restrict__ g, const bf16* __restrict__ b,
    bf16* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= n) return;
  const int64_t id = min(max(ids[j], 0), vocab - 1);
  const int64_t p = min(max(pos[j], 0), max_pos - 1);
  auto val = [&](int c) {
    return bf2f(word[id * d + c]) + bf2f(pemb[p * d + c]) + bf2f(temb[c]);
  };
  float s = 0.0f;
  for (int c = lane; c < d; c += 64) s += val(c);
  const float mean = wave_sum_f32(s) / (float)d;
  float v = 0.0f;
  for (int c = lane; c < d; c += 64) {
    const float t = val(c) - mean;
    v = fmaf(t, t, v);
  }
  const float r = 1.0f / sqrtf(wave_sum_f32(v) / (float)d + eps);
  bf16* o = out + (int64_t)j * d;
  for (int c = lane; c < d; c += 64) o[c] = f2bf((val(c) - mean) * r * bf2f(g[c]) + bf2f(b[c]));
}

// Early stop of a sequence (the computation ends once the state that feeds
// the classifier has exited): the flag of active row k is set when its
// sequence's [CLS] row (row b * seq_len) is flagged at this layer or is no
// longer active.  The list is ascending, so the [CLS] row, when active, is
// found by binary search; only the [CLS] row's own thread could write the
// flag that others read, and it writes back the value it read.
__global__ void cls_stop_kernel(const int32_t* __restrict__ act, const int32_t* __restrict__ n_act,
                                int max_n, int seq_len, uint8_t* __restrict__ flag) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  const int n = min(*n_act, max_n);
  if (k >= n) return;
  const int row = act[k];
  const int cls = row - row % seq_len;
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (act[mid] < cls) lo = mid + 1; else hi = mid;
  }
  const bool stop = lo >= n || act[lo] != cls || flag[lo] != 0;
  if (stop) flag[k] = 1;
}

// key_live[exited[k]] = 0 for k < min(*n_exited, max_n).
__global__ void mark_dead_kernel(const int32_t* __restrict__ exited,
                                 const int32_t* __restrict__ n_exited, int max_n,
                                 uint8_t* __restrict__ key_live) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < min(*n_exited, max_n)) key_live[exited[k]] = 0;
}

// One wave per (sequence, class): logits[b][c] = h_final[cls_b] . W[c] + bias[c],
// h_final = h[exit_layer & 1] of row cls_b = b * seq_len.
__global__ __launch_bounds__(64) void classify_head_kernel(
    int d, int n_classes, int seq_len, const bf16* __restrict__ h0, const bf16* __restrict__ h1,
    const int32_t* __restrict__ exit_layer, const bf16* __restrict__ w,
    const bf16* __restrict__ bias, float* __restrict__ logits) {
  const int b = blockIdx.x, c = blockIdx.y, lane = threadIdx.x;
  const int64_t row = (int64_t)b * seq_len;
  const bf16* h = ((exit_layer[row] & 1) ? h1 : h0) + row * d;
  float s = 0.0f;
  for (int k = lane; k < d; k += 64) s = fmaf(bf2f(h[k]), bf2f(w[(int64_t)c * d + k]), s);
  s = wave_sum_f32(s);
  if (lane == 0) logits[b * n_classes + c] = s + (bias ? bf2f(bias[c]) : 0.0f);
}

adept_status layernorm_rows(int d, float eps, const void* x, const int32_t* rows,
                            const int32_t* n_dev, int max_n, const void* g, const void* b,
                            void* out, hipStream_t s) {
  if (max_n <= 0) return ADEPT_OK;
  if (d % 8 == 0 && d <= 4096 && aligned16(x) && aligned16(out) && aligned16(g) && aligned16(b))
    return layernorm_rows_any(ADEPT_BF16, d, eps, x, x, nullptr, rows, n_dev, max_n, g, b, out,
                              true, s);
  ADEPT_LAUNCH(layernorm_kernel, dim3(ceil_div(max_n, 4)), dim3(256), 0, s, d, eps,
               (const bf16*)x, rows, n_dev, max_n, (const bf16*)g, (const bf16*)b, (bf16*)out);
  return launch_status("layernorm");
}

struct EncWs {
  void* compact; size_t compact_bytes;
  void* attend;  size_t attend_bytes;
  float* skinny; size_t skinny_bytes;
  size_t total;
};

EncWs carve(const adept_encoder_args* a, void* base) {
  EncWs w{};
  char* p = (char*)base;
  size_t off = 0;
  const int dq = a->n_heads * a->head_dim;
  w.compact_bytes = adept_compact_workspace_bytes(a->n_tok);
  w.compact = p + off; off += align256(w.compact_bytes);
  w.attend_bytes = attend_workspace_bytes(a->n_tok, a->n_seq, a->n_heads, a->head_dim, a->seq_len);
  w.attend = p + off; off += align256(w.attend_bytes);
  if (a->n_tok <= 64) {
    w.skinny_bytes = std::max({skinny_ws_bytes(3 * dq, a->d_model), skinny_ws_bytes(a->d_model, dq),
                               skinny_ws_bytes(a->d_ff, a->d_model),
                               skinny_ws_bytes(a->d_model, a->d_ff)});
    w.skinny = (float*)(p + off);
    off += align256(w.skinny_bytes);
  }
  w.total = off;
  return w;
}

const void* off(const void* base, int64_t elems) {
  return (const char*)base + elems * (int64_t)sizeof(bf16);
}

}  // namespace
}  // namespace adept

using namespace adept;

extern "C" size_t adept_encoder_workspace_bytes(const adept_encoder_args* a) {
  if (!a) return 0;
  return carve(a, nullptr).total;
}

extern "C" adept_status adept_encoder_embed(int n, int d_model, int vocab, int max_pos,
                                            float eps, const int32_t* ids, const int32_t* pos,
                                            const void* word_emb, const void* pos_emb,
                                            const void* type_emb, const void* ln_g,
                                            const void* ln_b, void* out, void* stream) {
  ADEPT_REQUIRE(n >= 0 && d_model > 0 && vocab > 0 && max_pos > 0, "encoder_embed: bad sizes");
  ADEPT_REQUIRE(ids && pos && word_emb && pos_emb && type_emb && ln_g && ln_b && out,
                "encoder_embed: NULL tensor");
  if (n == 0) return ADEPT_OK;
  ADEPT_LAUNCH(encoder_embed_kernel, dim3(ceil_div(n, 4)), dim3(256), 0, as_stream(stream), n,
               d_model, vocab, max_pos, eps, ids, pos, (const bf16*)word_emb, (const bf16*)pos_emb,
               (const bf16*)type_emb, (const bf16*)ln_g, (const bf16*)ln_b, (bf16*)out);
  return launch_status("encoder_embed");
}

extern "C" adept_status adept_classify_head(int n_seq, int seq_len, int d_model, int n_classes,
                                            const void* h0, const void* h1,
                                            const int32_t* exit_layer, const void* w_cls,
                                            const void* b_cls, float* logits, void* stream) {
  ADEPT_REQUIRE(n_seq >= 0 && seq_len > 0 && d_model > 0 && n_classes > 0,
                "classify_head: bad sizes");
  ADEPT_REQUIRE(h0 && h1 && exit_layer && w_cls && logits, "classify_head: NULL tensor");
  if (n_seq == 0) return ADEPT_OK;
  ADEPT_LAUNCH(classify_head_kernel, dim3(n_seq, n_classes), dim3(64), 0, as_stream(stream),
               d_model, n_classes, seq_len, (const bf16*)h0, (const bf16*)h1, exit_layer,
               (const bf16*)w_cls, (const bf16*)b_cls, logits);
  return launch_status("classify_head");
}

extern "C" adept_status adept_encoder_layer_step(const adept_encoder_args* a, int layer,
                                                 void* stream) {
  ADEPT_REQUIRE(a != nullptr, "encoder_layer_step: args is NULL");
  ADEPT_REQUIRE(a->dtype == ADEPT_BF16, "encoder_layer_step: bf16 only");
  const int N = a->n_layers, D = a->d_model, H = a->n_heads, hd = a->head_dim, F = a->d_ff;
  const int dq = H * hd;
  ADEPT_REQUIRE(N >= 1 && layer >= 1 && layer <= N, "encoder_layer_step: layer %d outside 1..%d",
                layer, N);
  ADEPT_REQUIRE(a->exit.n_layers == N, "encoder_layer_step: exit.n_layers != n_layers");
  ADEPT_REQUIRE(D > 0 && H > 0 && F > 0 && (hd == 64 || hd == 128) && a->n_tok > 0 &&
                    a->n_seq > 0 && a->seq_len > 0 && a->n_tok == a->n_seq * a->seq_len,
                "encoder_layer_step: bad sizes (n_tok must be n_seq * seq_len, hd 64/128)");
  ADEPT_REQUIRE(a->w_qkv && a->b_qkv && a->w_o && a->b_o && a->ln1_g && a->ln1_b && a->w_in &&
                    a->b_in && a->w_out && a->b_out && a->ln2_g && a->ln2_b,
                "encoder_layer_step: NULL weight");
  ADEPT_REQUIRE(a->h[0] && a->h[1] && a->pos && a->seq && a->active[0] && a->active[1] &&
                    a->n_active[0] && a->n_active[1] && a->exited && a->n_exited &&
                    a->exit_layer && a->exit_flag && a->key_live && a->key_len && a->k_buf &&
                    a->v_buf && a->q_buf && a->attn_out && a->y_buf && a->ffn_act,
                "encoder_layer_step: NULL tensor");
  ADEPT_REQUIRE(a->exit.prompt_level == 0,
                "encoder_layer_step: the all-at-once variant is defined for prefill only");
  ADEPT_REQUIRE(a->exit.metric == ADEPT_SIM_LOCAL || a->inertia,
                "encoder_layer_step: GLOBAL/BOTH metrics need inertia");
  const size_t need = adept_encoder_workspace_bytes(a);
  if (need > 0 && (!a->workspace || a->workspace_bytes < need)) {
    set_error("encoder_layer_step: workspace of %zu bytes needed", need);
    return ADEPT_E_WORKSPACE;
  }
  const EncWs ws = carve(a, a->workspace);
  hipStream_t s = as_stream(stream);
  const int in = (layer - 1) & 1, out = layer & 1;
  const int li = layer - 1;
  const int32_t* act = a->active[in];
  const int32_t* nact = a->n_active[in];
  const int maxn = a->n_tok;

  // 1. Q/K/V + bias; K and V of row j into the layer's buffers at slot j
  GemmArgs g{};
  g.M_max = maxn; g.M_dev = nact; g.N = 3 * dq; g.K = D;
  g.A = a->h[in]; g.a_rows = act; g.lda = D;
  g.B = off(a->w_qkv, (int64_t)li * 3 * dq * D); g.ldb = D; g.epi = EPI_QKV;
  g.bias = off(a->b_qkv, (int64_t)li * 3 * dq);
  g.rows = act; g.head_dim = hd; g.d_q = dq;
  g.q_out = a->q_buf; g.k_cache = a->k_buf; g.v_cache = a->v_buf; g.name = "enc_gemm_qkv";
  g.skinny_ws = ws.skinny; g.skinny_ws_bytes = ws.skinny_bytes;
  ADEPT_TRY(gemm(ADEPT_BF16, g, s));
  // 2. bidirectional attention over the live rows of each sequence
  ADEPT_TRY(attend_dispatch(ADEPT_BF16, H, hd, 1.0f / sqrtf((float)hd), 0, a->q_buf, act, nact,
                            maxn, a->pos, a->seq, a->n_seq, a->k_buf, a->v_buf, a->seq_len,
                            a->key_len, a->key_live, a->attn_out, ws.attend, ws.attend_bytes,
                            true, s));
  // 3. y = h + o Wo^T + bo, then h1 = LN1(y) in place
  GemmArgs go{};
  go.M_max = maxn; go.M_dev = nact; go.N = D; go.K = dq;
  go.A = a->attn_out; go.lda = dq; go.B = off(a->w_o, (int64_t)li * D * dq); go.ldb = dq;
  go.epi = EPI_RESID; go.bias = off(a->b_o, (int64_t)li * D);
  go.C = a->y_buf; go.ldc = D; go.resid = a->h[in]; go.rows = act; go.name = "enc_gemm_o";
  go.skinny_ws = ws.skinny; go.skinny_ws_bytes = ws.skinny_bytes;
  ADEPT_TRY(gemm(ADEPT_BF16, go, s));
  ADEPT_TRY(layernorm_rows(D, a->ln_eps, a->y_buf, act, nact, maxn, off(a->ln1_g, (int64_t)li * D),
                           off(a->ln1_b, (int64_t)li * D), a->y_buf, s));
  // 4. a = GELU(h1 W_in^T + b_in)
  GemmArgs gi{};
  gi.M_max = maxn; gi.M_dev = nact; gi.N = F; gi.K = D;
  gi.A = a->y_buf; gi.a_rows = act; gi.lda = D; gi.B = off(a->w_in, (int64_t)li * F * D);
  gi.ldb = D; gi.epi = EPI_GELU; gi.bias = off(a->b_in, (int64_t)li * F);
  gi.C = a->ffn_act; gi.ldc = F; gi.name = "enc_gemm_in";
  gi.skinny_ws = ws.skinny; gi.skinny_ws_bytes = ws.skinny_bytes;
  ADEPT_TRY(gemm(ADEPT_BF16, gi, s));
  // 5. h_out = LN2(h1 + a W_out^T + b_out)
  GemmArgs gu{};
  gu.M_max = maxn; gu.M_dev = nact; gu.N = D; gu.K = F;
  gu.A = a->ffn_act; gu.lda = F; gu.B = off(a->w_out, (int64_t)li * D * F); gu.ldb = F;
  gu.epi = EPI_RESID; gu.bias = off(a->b_out, (int64_t)li * D);
  gu.C = a->h[out]; gu.ldc = D; gu.resid = a->y_buf; gu.rows = act; gu.name = "enc_gemm_out";
  gu.skinny_ws = ws.skinny; gu.skinny_ws_bytes = ws.skinny_bytes;
  ADEPT_TRY(gemm(ADEPT_BF16, gu, s));
  ADEPT_TRY(layernorm_rows(D, a->ln_eps, a->h[out], act, nact, maxn,
                           off(a->ln2_g, (int64_t)li * D), off(a->ln2_b, (int64_t)li * D),
                           a->h[out], s));
  // 6. exit test (Eq. 7-8), active-list update, exited keys leave the key set
  ADEPT_TRY(adept_exit_test(ADEPT_BF16, D, layer, &a->exit, act, nact, maxn, a->h[out], a->h[in],
                            a->inertia, a->force_layer, a->exit_flag, a->sim_out, stream));
  if (a->cls_stop && maxn > 0) {
    ADEPT_LAUNCH(cls_stop_kernel, dim3(ceil_div(maxn, 256)), dim3(256), 0, s, act, nact, maxn,
                 a->seq_len, a->exit_flag);
    ADEPT_CHECK_LAUNCH("cls_stop");
  }
  ADEPT_TRY(adept_compact(layer, a->n_layers, a->exit_flag, act, nact, maxn, a->active[out],
                          a->n_active[out],
                          a->exited, a->n_exited, a->exit_layer, ws.compact, ws.compact_bytes,
                          stream));
  ADEPT_LAUNCH(mark_dead_kernel, dim3(ceil_div(maxn, 256)), dim3(256), 0, s, a->exited,
               a->n_exited, maxn, a->key_live);
  return launch_status("mark_dead");
}
