/*
 * adept.h -- C ABI of the MI355X (gfx950) hot path of ADEPT's token-level
 * early-exit forward pass (arXiv 2601.03700).
 *
 * Conventions (apply to every entry point)
 *  - Pointers are DEVICE pointers unless marked (host).  The caller owns all
 *    memory; the library never allocates or frees device memory (the one
 *    fixed scratch array of adept_kv_generate_noalloc is static).  Scratch
 *    space is passed in as `workspace` of at least the size returned by the
 *    matching *_workspace_bytes() query.
 *  - Calls only enqueue work on `stream` (a hipStream_t; NULL = the null
 *    stream) and return.  Variable counts (active rows, exited rows) live in
 *    device int32 cells; `max_*` host integers bound the launch grids and the
 *    kernels stop at the device count, so no call reads device memory back.
 *  - Shapes, enum values and pointer alignment (16 bytes for tensors) are
 *    validated on the host before anything is enqueued; on an error nothing
 *    is launched and the call returns a negative adept_status.
 *    adept_last_error() returns a message for the calling thread's last error.
 *  - Layers are numbered 1..N as in the paper (Section 3).  A token that exits
 *    at layer i* ran layers 1..i* in full; layers i*+1..N are "skipped".
 *    exit_layer[j] == N means token j never exited.
 *  - Per-token tensors are in token-row order [n_tok][...]; with a [B, T]
 *    prompt batch, row j = b*T + p (Appendix I flattens a batch this way).
 *    Index lists (int32) select rows; lists produced here are ascending.
 *  - Element types: ADEPT_F32 (float) or ADEPT_BF16 (bfloat16 stored as
 *    uint16).  Inertia is always float, similarities double.
 *  - Caches K and V are [N][n_slots][H][hd]; a token's slot is
 *    b * s_max + p (sequence b, position p).
 */
#ifndef ADEPT_H
#define ADEPT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ADEPT_ABI_VERSION 6

typedef enum {
  ADEPT_OK = 0,
  ADEPT_E_INVALID = -1,     /* bad argument; nothing enqueued */
  ADEPT_E_UNSUPPORTED = -2, /* valid but not implemented for these shapes/types */
  ADEPT_E_WORKSPACE = -3,   /* workspace missing or too small */
  ADEPT_E_HIP = -4          /* a HIP launch or runtime call failed */
} adept_status;

typedef enum { ADEPT_F32 = 0, ADEPT_BF16 = 1 } adept_dtype;

/* Decoder family of adept_layer_step (the paper's base models, Section 5):
 * LLAMA: RMSNorm, rotary positions, SwiGLU FFN, no biases;
 * GPT2: LayerNorm with bias, learned absolute positions (added by
 * adept_embed_positions), tanh-GELU MLP, biases on every projection, LM head
 * tied to the token embedding (the GPT2-XL shape). */
typedef enum { ADEPT_FAMILY_LLAMA = 0, ADEPT_FAMILY_GPT2 = 1 } adept_family;

/* Exit metric: GLOBAL compares h_i with the inertia of Section 4.1 (Eq. 7-8);
 * LOCAL compares h_i with h_{i-1} (the "local" metric of Appendix H.3);
 * BOTH is the combination Appendix H.3 compares the two against, which it
 * does not define: taken here as exit iff both cosines reach delta (the
 * inertia is kept and updated as for GLOBAL). */
typedef enum { ADEPT_SIM_GLOBAL = 0, ADEPT_SIM_LOCAL = 1, ADEPT_SIM_BOTH = 2 } adept_metric;

/* (host) Exit policy of Section 4.1, Eq. 8: token j exits at layer i iff
 * min_exit_layer <= i <= n_layers-1 and cos >= delta.  An undefined cosine
 * (a zero-norm vector, e.g. the empty inertia at layer 1) never exits, and
 * delta = +INFINITY never fires.  prompt_level = 1 selects the all-at-once
 * variant of Appendix H.2 for prefill passes (adept_exit_prompt_level): the
 * last prompt token of each sequence decides for all of its tokens; it is
 * honoured by adept_layer_step with attn_tiles = 1 and rejected by the
 * encoder step.  0 is the token-level method. */
typedef struct {
  double delta;
  int32_t min_exit_layer;
  int32_t n_layers;
  int32_t metric; /* adept_metric */
  int32_t prompt_level;
} adept_exit_cfg;

int adept_abi_version(void);
const char* adept_last_error(void);

/* Rotary table used by every kernel that applies RoPE: cos_out/sin_out are
 * [max_pos][head_dim/2] float, entry (p, k) = cos/sin(p * theta^(-2k/head_dim)),
 * with the angle formed in double precision on the device.  (The paper's base
 * models use rotary positions; the paper itself does not define them.) */
adept_status adept_rope_table(int max_pos, int head_dim, double theta,
                              float* cos_out, float* sin_out, void* stream);

/* ---------------------------------------------------------------------------
 * adept_exit_test -- the token-level exit policy (Section 4.1, Eq. 7-8;
 * Appendix H.3 for the local variant), for the active rows at layer `layer`.
 *
 *  active_rows[k], k < *n_active (device count, <= max_active): rows tested.
 *  h_cur  [n_tok][d_model] (dtype): h_i, the residual stream after layer i.
 *  h_prev [n_tok][d_model] (dtype): h_{i-1}; read only for ADEPT_SIM_LOCAL
 *         and ADEPT_SIM_BOTH (may be NULL otherwise).
 *  inertia [n_tok][d_model] float: Eq. 7's running sum of unit states of the
 *         layers before i.  For ADEPT_SIM_GLOBAL and ADEPT_SIM_BOTH it is read
 *         for the test and then updated in place, inertia += h_i/|h_i| (after
 *         the test).  For LOCAL it is not touched (may be NULL).
 *  force_layer [n_tok] int32, nullable: f = force_layer[row] > 0 replaces the
 *         policy for that row by "exit iff layer == f and layer <= N-1"; 0
 *         keeps the policy (teacher forcing and fixed exit schedules).
 *  exit_flag [max_active] uint8 out: 1 = exit, aligned with active_rows.
 *  sim_out [max_active] double out, nullable: the cosine (NaN if undefined);
 *         for BOTH the smaller of the two cosines (NaN if either is).
 *
 * The three sums <h,h>, <r,r>, <h,r> are reduced in double precision from
 * the stored values (each product is exact in double), the decision is
 * taken in double.  One wavefront per row; HBM-bound.  d_model must be a
 * multiple of 4 (GLOBAL, BOTH, and LOCAL f32) or 8 (LOCAL bf16) and at most
 * 8192 (GLOBAL; 8192 f32 / 16384 bf16 for LOCAL; 4096 for BOTH), else
 * ADEPT_E_INVALID / ADEPT_E_UNSUPPORTED; h_cur, h_prev and the inertia
 * 16-byte aligned.
 * ------------------------------------------------------------------------- */
adept_status adept_exit_test(adept_dtype dt, int d_model, int layer, const adept_exit_cfg* cfg,
                             const int32_t* active_rows, const int32_t* n_active, int max_active,
                             const void* h_cur, const void* h_prev, float* inertia,
                             const int32_t* force_layer, uint8_t* exit_flag, double* sim_out,
                             void* stream);

/* ---------------------------------------------------------------------------
 * adept_exit_prompt_level -- the all-at-once variant of Appendix H.2: after
 * adept_exit_test, every active row takes the decision of its sequence's
 * last prompt token, i.e. the active row of that sequence with the largest
 * position, so a sequence's tokens exit together.
 *
 *  active_rows[k], k < *n_active (<= max_active); exit_flag[k] in/out.
 *  seq [n_tok] int32: sequence of each row, 0 <= seq < n_seq (rows outside
 *  that range keep their flag); pos [n_tok] int32 >= 0.
 *  workspace: adept_exit_prompt_level_workspace_bytes(n_seq) bytes, 8-byte
 *  aligned (one 64-bit key per sequence), else ADEPT_E_WORKSPACE.
 *  Three small kernels: clear the keys, per sequence the largest
 *  (position, index) key, then the broadcast.
 * ------------------------------------------------------------------------- */
size_t adept_exit_prompt_level_workspace_bytes(int n_seq);
adept_status adept_exit_prompt_level(const int32_t* active_rows, const int32_t* n_active,
                                     int max_active, const int32_t* seq, const int32_t* pos,
                                     int n_seq, uint8_t* exit_flag, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * adept_hsm_forward -- the Hidden State Mapper of Section 4.2 (Appendix B,
 * Table S1, Fig. S1): the mapped state s~ of each exiting token from its
 * current state s_i, its previous state s_{i-1} and the inertia of Eq. 7
 * (as the exit test of layer i saw it).  Per row (D = d_model):
 *   x_r = RMSNorm(z_r) * g0 for z = (s_i, s_{i-1}, inertia), r = 0, 1, 2
 *   u   = conv_bias + sum_{r,t} conv[r][t] * x_r[d + t - 1]  (zero outside 0..D-1)
 *   a   = W1 u + b1                  [4D]
 *   c   = W3 gelu(W2 gelu(a) + b2) + b3   (gelu: exact erf form)
 *   e   = W4 (RMSNorm(c) * g1 + a) + b4   [D]
 *   s~  = RMSNorm(e) * g2 + u
 * (The paper leaves the activations, the skip sources and the biases open;
 * this is the reading implemented.)  The four layers run as MFMA GEMMs.
 *
 *  rows[k], k < *n_rows (<= max_rows): token rows of the inputs.
 *  h_cur, h_prev [n_tok][D] bf16; inertia [n_tok][D] float.
 *  inertia_updated: 1 when the inertia already holds layer i's update
 *  (inertia += s_i/|s_i|, the exit test's order), which is then taken back;
 *  0 when it is the inertia before layer i.
 *  out [n_tok][D] bf16: out[rows[k]] = s~_k; may be h_cur itself.
 *  Weights (bf16, device, 16-byte aligned matrices in [out][in] order):
 *  W1 [4D][D], W2 [8D][4D], W3 [4D][8D], W4 [D][4D], biases b1..b4, gains
 *  g0 [D], g1 [4D], g2 [D]; the convolution (host floats) by value.
 *  d_model a multiple of 256; workspace adept_hsm_workspace_bytes(D,
 *  max_rows) bytes (44 * D bytes per row), 16-byte aligned.
 * ------------------------------------------------------------------------- */
typedef struct {
  const void* g0;
  float conv[3][3];      /* (host) row: state (current, previous, inertia); column: offset -1..1 */
  float conv_bias;       /* (host) */
  const void* w1; const void* b1;
  const void* w2; const void* b2;
  const void* w3; const void* b3;
  const void* g1;
  const void* w4; const void* b4;
  const void* g2;
} adept_hsm_weights;
size_t adept_hsm_workspace_bytes(int d_model, int max_rows);
adept_status adept_hsm_forward(adept_dtype dt, int d_model, float eps, const adept_hsm_weights* w,
                               const int32_t* rows, const int32_t* n_rows, int max_rows,
                               const void* h_cur, const void* h_prev, const float* inertia,
                               int inertia_updated, void* out, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * adept_compact -- the active-index update of Appendix I: split the active
 * list by the exit flags into the rows that continue and the rows that exit.
 *
 *  exit_flag[k], active_rows[k] for k < *n_active.
 *  next_rows / *n_next out: rows with flag 0, in the order of active_rows.
 *  exited_rows / *n_exited out: rows with flag 1, same order.
 *  exit_layer [n_tok] int32: exit_layer[row] = layer for every exited row;
 *  every listed row that continues must hold n_layers (never exited, as
 *  adept_token_init sets it): the multi-pass form writes dense stretches of
 *  the list (64 consecutive rows) as whole lines, n_layers included.
 *  Counts are exact; with an ascending active list both outputs are ascending.
 *  next_rows / exited_rows must not alias active_rows.
 *  workspace: adept_compact_workspace_bytes(max_active) bytes, 8-byte aligned
 *  (0 bytes, workspace may be NULL, for max_active <= 65536); larger lists
 *  keep per-16K-entry exit counts and one 64-bit exit mask per 64 entries
 *  there.  ADEPT_E_WORKSPACE if it is missing or too small.
 * ------------------------------------------------------------------------- */
size_t adept_compact_workspace_bytes(int max_active);
adept_status adept_compact(int layer, int n_layers, const uint8_t* exit_flag,
                           const int32_t* active_rows,
                           const int32_t* n_active, int max_active, int32_t* next_rows,
                           int32_t* n_next, int32_t* exited_rows, int32_t* n_exited,
                           int32_t* exit_layer, void* workspace, size_t workspace_bytes,
                           void* stream);

/* ---------------------------------------------------------------------------
 * adept_kv_generate -- decoupled KV generation (Section 4, Eq. 6; Section
 * 4.3, Eq. 9): for every listed row j and every skipped layer r with
 * exit_layer[j] < r <= n_layers, with s = s_map[j] (the mapped state s~):
 *     u   = RMSNorm_r(s) = s / sqrt(mean(s^2) + eps) * attn_gain[r]
 *     K[r][cache_slot[j]] = RoPE(u Wk_r^T, pos[j]),   V[r][cache_slot[j]] = u Wv_r^T
 * All (token, layer) pairs are computed in one grouped GEMM, with no
 * layer-sequential dependency.
 *
 *  s_map [n_tok][d_model] (dtype); rows[k], k < *n_rows (<= max_rows).
 *  exit_layer, cache_slot, pos: [n_tok] int32.
 *  w_kv: layer r's block starts at w_kv + (r-1)*w_kv_layer_stride elements and
 *        is [2*H*hd][d_model] (nn.Linear order): H*hd rows of Wk_r, then H*hd
 *        rows of Wv_r.  (A stacked [N][3*H*hd][D] QKV weight passes its K part
 *        with stride 3*H*hd*D.)
 *  attn_gain [n_layers][d_model] (dtype), nullable: layer r's pre-attention
 *        RMSNorm gain.  NULL means the gains are already folded into the
 *        columns of w_kv (adept_fold_gain), which the bf16 path requires; the
 *        kernels then apply only the 1/rms(s) row factor.
 *  rope_cos/rope_sin [rope_max_pos][hd/2] float (adept_rope_table).
 *  k_cache/v_cache [n_layers][n_slots][H][hd] (dtype): written only at the
 *        (layer, slot) pairs above.
 * bf16 requires d_model % 64 == 0 and head_dim in {64, 128}.
 * ------------------------------------------------------------------------- */
size_t adept_kv_generate_workspace_bytes(int n_layers, int max_rows);
adept_status adept_kv_generate(adept_dtype dt, int n_layers, int d_model, int n_heads,
                               int head_dim, float eps, const void* s_map, const int32_t* rows,
                               const int32_t* n_rows, int max_rows, const int32_t* exit_layer,
                               const int32_t* cache_slot, const int32_t* pos, const void* w_kv,
                               int64_t w_kv_layer_stride, const void* attn_gain,
                               const float* rope_cos, const float* rope_sin, int rope_max_pos,
                               void* k_cache, void* v_cache, int64_t n_slots, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * adept_kv_generate_layernorm -- decoupled KV generation (Section 4, Eq. 6;
 * Section 4.3, Eq. 9) for the LayerNorm family: for every listed row j and
 * every skipped layer r with exit_layer[j] < r <= n_layers, s = s_map[j]:
 *     xh  = (s - mean(s)) / sqrt(var(s) + eps)            (no affine part)
 *     K[r][cache_slot[j]] = xh Wk'_r^T + bk'_r,   V[r][cache_slot[j]] = xh Wv'_r^T + bv'_r
 * where W'_r carries layer r's LayerNorm gain in its columns and b'_r its
 * shift, b'_r = b_r + W_r beta_r (adept_fold_gain, adept_fold_bias): this is
 * layer r's own LayerNorm and K/V projection applied to s.  No RoPE (the
 * family's positions enter through the embedding).  One grouped GEMM.
 *
 *  w_kv: layer r's block at w_kv + (r-1)*w_kv_layer_stride elements,
 *        [2*H*hd][d_model] (K rows then V rows); b_kv: layer r's [2*H*hd] bias
 *        at b_kv + (r-1)*b_kv_layer_stride.  Other arguments as for
 *        adept_kv_generate.  bf16; d_model % 64 == 0, H*hd % 32 == 0;
 *  workspace: adept_kv_generate_layernorm_workspace_bytes(n_layers, max_rows,
 *        d_model) bytes (the plan plus the normalised rows), 16-byte aligned.
 * ------------------------------------------------------------------------- */
size_t adept_kv_generate_layernorm_workspace_bytes(int n_layers, int max_rows, int d_model);
adept_status adept_kv_generate_layernorm(adept_dtype dt, int n_layers, int d_model, int n_heads,
                                         int head_dim, float eps, const void* s_map,
                                         const int32_t* rows, const int32_t* n_rows, int max_rows,
                                         const int32_t* exit_layer, const int32_t* cache_slot,
                                         const void* w_kv, int64_t w_kv_layer_stride,
                                         const void* b_kv, int64_t b_kv_layer_stride,
                                         void* k_cache, void* v_cache, int64_t n_slots,
                                         void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * adept_kv_generate_noalloc -- adept_kv_generate for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc): same arguments and results, minus the
 * workspace.  Its scratch (exit-layer plan, work list and counters, sorted
 * rows, row scales) is a fixed 4 MiB device array inside the library, one
 * copy per GPU, held until the process ends; the call allocates nothing.
 * adept_kv_generate_workspace_bytes(n_layers, max_rows) must not exceed
 * 4 MiB (32 layers: up to about 480K rows), else ADEPT_E_UNSUPPORTED and
 * nothing is enqueued.  Every call on a GPU uses that GPU's one array and
 * re-initialises what it reads, so calls that overlap on one GPU (other
 * streams, other host threads) race: serialise them.  The device current
 * at the call selects the array; the first call on a device looks up its
 * address (ADEPT_E_HIP if that fails).
 * ------------------------------------------------------------------------- */
adept_status adept_kv_generate_noalloc(adept_dtype dt, int n_layers, int d_model, int n_heads,
                                       int head_dim, float eps, const void* s_map,
                                       const int32_t* rows, const int32_t* n_rows, int max_rows,
                                       const int32_t* exit_layer, const int32_t* cache_slot,
                                       const int32_t* pos, const void* w_kv,
                                       int64_t w_kv_layer_stride, const void* attn_gain,
                                       const float* rope_cos, const float* rope_sin,
                                       int rope_max_pos, void* k_cache, void* v_cache,
                                       int64_t n_slots, void* stream);

/* ---------------------------------------------------------------------------
 * adept_attend -- attention of the active tokens over one layer's cache,
 * whose entries are computed (tokens still active at this layer) or
 * generated (tokens that exited earlier) (Section 3, Eq. 5; Section 4.3).
 *
 *  q [max_active][H][hd] (dtype): compacted queries; entry k is for row rows[k].
 *  rows[k], k < *n_active.  seq[row] must be non-decreasing in k.
 *  pos, seq [n_tok] int32: position and sequence of each row.
 *  k_layer/v_layer: this layer's cache, [n_seq*s_max][H][hd] (dtype).
 *  causal=1: entry k attends to slots seq*s_max + t, t = 0..pos[rows[k]].
 *  causal=0: t = 0..key_len[seq]-1 (bidirectional), key_len [n_seq] int32.
 *  key_live [n_seq*s_max] uint8, nullable: keys with 0 are left out.
 *  out [max_active][H][hd] (dtype): softmax(q K^T * scale) V per head, with
 *      f32 scores and softmax statistics.
 *  workspace: adept_attend_workspace_bytes(max_active, n_seq, H, hd, s_max)
 *      bytes (at most about 17 MB), 16-byte aligned; nullable, but then bf16
 *      takes the slow generic kernel.  bf16 with hd 64/128 uses query tiles on
 *      MFMA when the queries average at least 4 per sequence (prefill,
 *      classification), otherwise key chunks streamed per (query, head) and
 *      merged (decode).
 * ------------------------------------------------------------------------- */
size_t adept_attend_workspace_bytes(int max_active, int n_seq, int n_heads, int head_dim,
                                    int s_max);
adept_status adept_attend(adept_dtype dt, int n_heads, int head_dim, float scale, int causal,
                          const void* q, const int32_t* rows, const int32_t* n_active,
                          int max_active, const int32_t* pos, const int32_t* seq, int n_seq,
                          const void* k_layer, const void* v_layer, int s_max,
                          const int32_t* key_len, const uint8_t* key_live, void* out,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Whole-layer orchestration of the generative path (Appendix I):
 * adept_layer_step(layer=i) enqueues, for the rows of active[(i-1)&1]
 * (LLAMA family; GPT2: LayerNorm for the norms, biased projections without
 * RoPE, tanh-GELU MLP, adept_kv_generate_layernorm for the generation):
 *   RMSNorm -> QKV GEMM (+RoPE; own K/V into cache[i]) -> adept_attend ->
 *   O GEMM (+residual: h[i&1] = h[(i-1)&1] + o Wo^T) -> RMSNorm ->
 *   gate/up GEMM (+SwiGLU) -> down GEMM (+residual) -> adept_exit_test ->
 *   adept_compact (next list into active[i&1], exited rows into `exited`) ->
 *   [adept_hsm_forward on the exited rows, when `hsm` is set] ->
 *   adept_kv_generate for the rows exited at i (layers i+1..N); with
 *   attn_tiles = 0 (decode) the generation of every exited row is enqueued
 *   once, by the step of layer N, after copying the exit states into h[N&1]
 *   (or, with kv_fused, done by the QKV GEMM of each later layer).
 * The residual stream ping-pongs between h[0] and h[1]: a token's final
 * state is h[exit_layer & 1][row] (its state at exit, the identity mapped
 * state).  Before layer 1 the caller puts h_0 in h[0], zeroes the inertia,
 * fills active[0] with the rows, *n_active[0] = count and exit_layer = N.
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t dtype;        /* adept_dtype */
  int32_t n_layers, d_model, n_heads, head_dim, d_ff;
  float rms_eps;
  adept_exit_cfg exit;
  /* weights, stacked over layers (dtype).  The pre-norm gains are folded
   * into the matrices that consume the normalised input (adept_fold_gain):
   * w_qkv columns carry the layer's attention-norm gain, w_gate / w_up
   * columns its FFN-norm gain; the kernels apply only the 1/rms row factor. */
  const void* w_qkv;     /* [N][3*H*hd][D]: Wq rows, Wk rows, Wv rows (gain folded) */
  const void* w_o;       /* [N][D][H*hd] */
  const void* w_gate;    /* [N][F][D] (gain folded) */
  const void* w_up;      /* [N][F][D] (gain folded) */
  const void* w_down;    /* [N][D][F] */
  const float* rope_cos; /* [rope_max_pos][hd/2] */
  const float* rope_sin;
  int32_t rope_max_pos;
  /* token state */
  int32_t n_tok;         /* rows in the per-token tensors */
  int32_t max_active;    /* (host) bound on the active rows entering this layer */
  int32_t n_seq, s_max;
  int32_t attn_tiles;    /* 1: prompt rows (prefill): attention by query tiles, K/V of
                            the rows that exit at layer i generated right after layer i;
                            0: one row per sequence (decode): attention by key chunks,
                            K/V of all exited rows generated after layer N or, with
                            kv_fused, inside the later layers (no row of the pass
                            reads them); the pass must then run all N layers */
  void* h[2];            /* [n_tok][D] residual stream ping-pong */
  float* inertia;        /* [n_tok][D] (GLOBAL and BOTH metrics) */
  const int32_t* pos;    /* [n_tok] */
  const int32_t* seq;    /* [n_tok] */
  const int32_t* slot;   /* [n_tok] */
  int32_t* active[2];    /* [n_tok] each */
  int32_t* n_active[2];  /* device counts */
  int32_t* exited;       /* [n_tok] rows exited at this layer */
  int32_t* n_exited;     /* device count */
  int32_t* exit_layer;   /* [n_tok] */
  uint8_t* exit_flag;    /* [n_tok] */
  double* sim_out;       /* [n_tok] nullable, aligned with the active list */
  const int32_t* force_layer; /* [n_tok] nullable */
  void* k_cache;         /* [N][n_slots][H][hd] */
  void* v_cache;
  int64_t n_slots;
  /* per-layer scratch (dtype), caller-allocated */
  void* q_buf;           /* [n_tok][H*hd] */
  void* attn_out;        /* [n_tok][H*hd] */
  void* ffn_act;         /* [n_tok][F] */
  void* workspace;
  size_t workspace_bytes;
  /* mapper of the exiting rows (Section 4.2): NULL = identity (s~ = h_i);
   * else adept_hsm_forward maps the rows exited at layer i in place in
   * h[i&1] before their K/V are generated (bf16, GLOBAL or BOTH metric: it
   * reads the inertia) */
  const adept_hsm_weights* hsm;
  /* decoder family (adept_family).  GPT2 (bf16): rms_eps is the LayerNorm
   * eps; the layer norms run without their affine part, whose gains are
   * folded into w_qkv (LN1) and w_gate (LN2) and whose shifts into b_qkv and
   * b_fc; w_gate holds the MLP's first projection W_fc [N][F][D], w_down its
   * second W_proj [N][D][F], w_up and the rotary table are unused (NULL);
   * d_model, H*hd and F multiples of 64 */
  int32_t family;
  const void* b_qkv;    /* [N][3*H*hd] (GPT2) */
  const void* b_o;      /* [N][D] */
  const void* b_fc;     /* [N][F] */
  const void* b_proj;   /* [N][D] */
  /* decode passes (attn_tiles = 0), bf16: 1 = generate the K/V of exited rows
   * inside each later layer's QKV GEMM (the GEMM's rows are the active rows
   * followed by the rows that exited at a layer below it, each read from its
   * exit state; W_k / W_v are then read once per pass with no extra launch),
   * 0 = one grouped generation after layer N.  Same cache contents either way
   * (Eq. 6 leaves the order of the generation free). */
  int32_t kv_fused;
} adept_layer_args;

size_t adept_layer_workspace_bytes(const adept_layer_args* a);
adept_status adept_layer_step(const adept_layer_args* a, int layer, void* stream);

/* Folds a norm gain into the weight matrices that consume the normalised
 * vector, in place: w[l][o][c] *= gain[l][c] for l < n_mats, o < rows,
 * c < cols, rounded to dtype; matrix l starts at w + l*mat_stride, its gain at
 * gain + l*gain_stride (elements).  Since (x * g) W^T = x (W diag(g))^T, an
 * RMSNorm followed by a projection becomes a projection scaled per row by
 * 1/rms(x), which the GEMM epilogues apply.  Done once at model load. */
adept_status adept_fold_gain(adept_dtype dt, int n_mats, int rows, int cols, void* w,
                             int64_t mat_stride, const void* gain, int64_t gain_stride,
                             void* stream);

/* Folds a LayerNorm shift into the bias of the projection that consumes the
 * normalised vector, in place: bias[l][o] += sum_c w[l][o][c] * shift[l][c]
 * for l < n_mats, o < rows (w unfolded: run before adept_fold_gain), with
 * matrix l at w + l*mat_stride, its shift at shift + l*shift_stride and its
 * bias at bias + l*bias_stride (elements).  (xh g + beta) W^T + b =
 * xh (W diag g)^T + (b + W beta).  Done once at model load. */
adept_status adept_fold_bias(adept_dtype dt, int n_mats, int rows, int cols, const void* w,
                             int64_t mat_stride, const void* shift, int64_t shift_stride,
                             void* bias, int64_t bias_stride, void* stream);

/* Embedding with learned absolute positions (GPT2 family, before layer 1):
 * h0[k] = wte[ids[k]] + wpe[pos[k]] (ids and positions clamped into the
 * tables), wte [vocab][D], wpe [max_pos][D], h0 [n][D] (dtype). */
adept_status adept_embed_positions(adept_dtype dt, int n, int d_model, int vocab, int max_pos,
                                   const int32_t* ids, const int32_t* pos, const void* wte,
                                   const void* wpe, void* h0, void* stream);

/* Final LayerNorm (with gain and shift) and LM head of the GPT2 family, as
 * adept_final_logits: logits[k] = LN(h[exit_layer[row] & 1][row]; ln_g, ln_b)
 * lm_head^T (lm_head: the token embedding when tied).  bf16; d_model and
 * vocab multiples of 64. */
adept_status adept_final_logits_layernorm(adept_dtype dt, int d_model, int vocab, float eps,
                                          const void* h0_buf, const void* h1_buf,
                                          const int32_t* exit_layer, const int32_t* rows,
                                          const int32_t* n_rows, int max_rows, const void* ln_g,
                                          const void* ln_b, const void* lm_head, void* x_norm,
                                          float* logits, void* stream);

/* Embedding gather (support step before layer 1): h0[k] = embed[ids[k]],
 * k < n; embed [vocab][D] (dtype), h0 [n][D] (dtype). */
adept_status adept_embed(adept_dtype dt, int n, int d_model, int vocab, const int32_t* ids,
                         const void* embed, void* h0, void* stream);

/* Final norm and LM head (support step after layer N): for k < *n_rows,
 * row = rows[k]: logits[k] = RMSNorm(h[exit_layer[row] & 1][row]; final_norm)
 * lm_head^T, as float.  An exited token uses its state at exit (Fig. 1: the
 * mapped state is propagated to the end of the layer chain).
 * x_norm is [max_rows][D] (dtype) scratch. */
adept_status adept_final_logits(adept_dtype dt, int d_model, int vocab, float eps,
                                const void* h0_buf, const void* h1_buf,
                                const int32_t* exit_layer, const int32_t* rows,
                                const int32_t* n_rows, int max_rows, const void* final_norm,
                                const void* lm_head, void* x_norm, float* logits, void* stream);

/* State set-up before layer 1 of a token pass: active[k] = k and
 * exit_layer[k] = n_layers for k < n_tok, *n_active = n_tok, and the inertia
 * [n_tok][d_model] (nullable) zeroed (Eq. 7's sum starts empty). */
adept_status adept_token_init(int n_tok, int n_layers, int d_model, int32_t* active,
                              int32_t* n_active, int32_t* exit_layer, float* inertia,
                              void* stream);

/* Greedy next token: out[k] = argmax_v logits[k][v] for k < n, ties to the
 * lowest id (support step of the generation loop). */
adept_status adept_argmax(int n, int vocab, const float* logits, int32_t* out, void* stream);

/* ---------------------------------------------------------------------------
 * Classification mode (Section 4.3, downstream tasks): token-level exit in a
 * post-norm encoder (BERT-style: biases, LayerNorm, GELU, learned positions).
 * Exited tokens stop and leave the key set of every later layer; there is no
 * KV generation.  A sequence's output is its first ([CLS]) row at that row's
 * exit layer.  bf16 only.  Rows are j = b*seq_len + p for n_seq sequences.
 *
 * adept_encoder_layer_step(layer=i) enqueues, for the rows of
 * active[(i-1)&1]: QKV GEMM + bias (Q into q_buf, K/V into k_buf/v_buf at
 * row j) -> attention of each row over the rows of its sequence whose
 * key_live byte is 1 (bidirectional, keys < key_len[b]) -> O GEMM + bias +
 * residual into y_buf -> LayerNorm 1 (in place) -> GEMM + bias + GELU into
 * ffn_act -> GEMM + bias + residual into h[i&1] -> LayerNorm 2 (in place)
 * -> adept_exit_test -> [cls_stop: the flags of rows whose sequence's [CLS]
 * row exits here or has left are set] -> adept_compact -> key_live[row] = 0
 * for the rows that exited.  Before layer 1 the caller runs adept_encoder_embed into h[0],
 * adept_token_init, and sets key_live to 1 for every row.  A row's final
 * state is h[exit_layer & 1][row].
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t dtype;        /* ADEPT_BF16 */
  int32_t n_layers, d_model, n_heads, head_dim, d_ff;
  float ln_eps;
  adept_exit_cfg exit;
  /* weights stacked over layers, nn.Linear [out][in] order (bf16) */
  const void* w_qkv;    /* [N][3*H*hd][D]: Wq rows, Wk rows, Wv rows */
  const void* b_qkv;    /* [N][3*H*hd] */
  const void* w_o;      /* [N][D][H*hd] */
  const void* b_o;      /* [N][D] */
  const void* ln1_g;    /* [N][D] */
  const void* ln1_b;    /* [N][D] */
  const void* w_in;     /* [N][F][D] */
  const void* b_in;     /* [N][F] */
  const void* w_out;    /* [N][D][F] */
  const void* b_out;    /* [N][D] */
  const void* ln2_g;    /* [N][D] */
  const void* ln2_b;    /* [N][D] */
  int32_t n_tok, n_seq, seq_len;   /* n_tok = n_seq * seq_len */
  int32_t cls_stop;     /* 1: a row also leaves at the layer where its sequence's
                           [CLS] row exits (or at once if that row is no longer
                           active): the output no longer depends on it */
  void* h[2];            /* [n_tok][D] residual stream ping-pong */
  float* inertia;        /* [n_tok][D] (GLOBAL and BOTH metrics) */
  const int32_t* pos;    /* [n_tok] position of row j (j mod seq_len) */
  const int32_t* seq;    /* [n_tok] sequence of row j */
  int32_t* active[2];    /* [n_tok] ping-pong active lists */
  int32_t* n_active[2];  /* device counts */
  int32_t* exited;       /* [n_tok] rows that exited at this layer */
  int32_t* n_exited;
  int32_t* exit_layer;   /* [n_tok] */
  uint8_t* exit_flag;    /* [n_tok] */
  double* sim_out;       /* [n_tok] nullable */
  const int32_t* force_layer;  /* [n_tok] nullable, as in adept_exit_test */
  uint8_t* key_live;     /* [n_tok]: 1 while the row is a key (not exited) */
  const int32_t* key_len;      /* [n_seq] keys per sequence (normally seq_len) */
  void* k_buf;           /* [n_tok][H*hd] this layer's K of the active rows */
  void* v_buf;           /* [n_tok][H*hd] */
  void* q_buf;           /* [n_tok][H*hd] (compact order) */
  void* attn_out;        /* [n_tok][H*hd] (compact order) */
  void* y_buf;           /* [n_tok][D] attention sub-layer output */
  void* ffn_act;         /* [n_tok][F] (compact order) */
  void* workspace;       /* adept_encoder_workspace_bytes(), 256-byte aligned */
  size_t workspace_bytes;
} adept_encoder_args;

size_t adept_encoder_workspace_bytes(const adept_encoder_args* a);
adept_status adept_encoder_layer_step(const adept_encoder_args* a, int layer, void* stream);

/* h0[j] = LayerNorm(word_emb[ids[j]] + pos_emb[pos[j]] + type_emb) * ln_g + ln_b
 * (token type 0 for every row; f32 statistics; ids and positions clamped
 * into the tables).  word_emb [vocab][D], pos_emb [max_pos][D], type_emb,
 * ln_g, ln_b [D], out [n][D] (bf16). */
adept_status adept_encoder_embed(int n, int d_model, int vocab, int max_pos, float eps,
                                 const int32_t* ids, const int32_t* pos, const void* word_emb,
                                 const void* pos_emb, const void* type_emb, const void* ln_g,
                                 const void* ln_b, void* out, void* stream);

/* Linear head on each sequence's [CLS] row at its exit (Section 4.3):
 * logits[b][c] = h[exit_layer[r] & 1][r] . w_cls[c] + b_cls[c], r = b*seq_len.
 * w_cls [n_classes][D], b_cls [n_classes] nullable (bf16); logits f32. */
adept_status adept_classify_head(int n_seq, int seq_len, int d_model, int n_classes,
                                 const void* h0, const void* h1, const int32_t* exit_layer,
                                 const void* w_cls, const void* b_cls, float* logits,
                                 void* stream);

/* Kernel timing for measurement runs.  While enabled, every kernel the
 * library launches is bracketed by two HIP events on its own stream, and
 * adept_timing_get() (which waits for the pending events) reports, per
 * kernel name, the launch count and the summed elapsed milliseconds.
 * Names are sorted; index 0..adept_timing_count()-1.  No device memory is
 * used.  Disabled by default; reset clears the totals. */
adept_status adept_timing_enable(int on);
/* Restricts the bracketing to launches whose kernel name starts with `prefix`
 * (host string, copied); NULL or "" times every launch again (the default). */
adept_status adept_timing_select(const char* prefix);
void adept_timing_reset(void);
int adept_timing_count(void);
adept_status adept_timing_get(int idx, char* name, int name_len, int64_t* launches,
                              double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* ADEPT_H */
