"""CPU oracle of ADEPT's token-level early-exit forward pass (fp64, numpy).

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that the
HIP path is checked against.  Only the test suite, the package smoke check
and the bench's CPU-baseline leg may import it; the product path never calls
it and shares no code with it.

Everything is computed in float64 from the (float32 / bfloat16-valued) seeded
inputs.  The paper fixes no precision, so fp64 is the reference arithmetic;
the one place where floating point decides an integer (the exit decision) is
also taken in fp64, which is the precision the GPU exit test reduces in.

Notation follows the paper: layers are numbered i = 1..N (Section 3, state
space); token j's hidden state after layer i is s^h_{i,j}, written h_i here;
h_0 is the embedding.  "Exit at i*" means layers 1..i* run in full and the
skipped layers r = i*+1..N only receive generated keys/values (Section 4,
Eq. 6; Section 4.3, Eq. 9).

Readings of the paper taken here (where it is silent or ambiguous):
  * inertia at layer i is the sum of the unit-normalised states of layers
    1..i-1 (Eq. 7); the test at layer i compares h_i with it and the update
    with h_i happens after the test.  At i = 1 the sum is empty, the cosine
    is 0/0 = NaN and the token continues.
  * the test runs only for i_min <= i <= N-1 (exiting at N skips nothing).
  * the mapped state s~ fed to the KV generation is the identity map of the
    exit state, s~ = h_{i*}, unless a mapper is given (the paper's trained
    mapper is not available; oracle/hsm.py holds its architecture, which
    takes the inertia as the exit test of layer i* saw it).
  * generated K/V of layer r apply layer r's own pre-attention RMSNorm, its
    own K/V projection and, for K, the rotary embedding at the token's
    position -- i.e. s~ is treated as layer r's input (Eq. 9).
  * generated entries are visible to every active token's attention at the
    layers after the exit (Section 4.3; Appendix I), so K/V of tokens that
    exit at layer i are written before the attention of layer i+1.
  * an exited token's final state is its mapped state (Fig. 1 caption), so
    its logits use h_{i*}.
  * compaction keeps both lists in ascending row order (Appendix I update).
  * the "local" metric of Appendix H.3 is cos(h_i, h_{i-1}).
  * the "both" metric of Appendix H.3 (not defined there) exits only when
    the global and the local cosine both reach delta; its similarity is
    the smaller of the two, and the inertia is kept as for the global one.
  * the GPT-2-style family (Section 5's GPT2-XL): Eq. 9 applies layer r's
    first LayerNorm (gain and shift) and its biased K/V projections to s~;
    positions enter through the learned position embedding only, so no
    rotation is applied to generated keys.
  * classification (Section 4.3): exited tokens leave the key set of later
    layers and, once a sequence's [CLS] row has exited, its other rows stop
    with it (the classifier only reads that row).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

F64 = np.float64

GPT2 = "gpt2"       # decoder family: LayerNorm with bias, learned positions, GELU, biases

GLOBAL = "global"   # inertia metric, Section 4.1 Eq. 7-8
LOCAL = "local"     # consecutive-layer metric, Appendix H.3
BOTH = "both"       # both of them (Appendix H.3 names the combination, not its rule)


# ---------------------------------------------------------------------------
# Building blocks of the base model (not the paper's contribution; the base
# model is a Llama-style pre-norm decoder used in inference mode, Section 5).
# ---------------------------------------------------------------------------

def rms_norm(x, gain, eps):
    """y = x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    x = np.asarray(x, F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, F64)


def layer_norm(x, gain, bias, eps):
    """(x - mean) / sqrt(var + eps) * gain + bias over the last axis."""
    x = np.asarray(x, F64)
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(gain, F64) + np.asarray(bias, F64)


def rope_cos_sin(pos, head_dim, theta):
    """cos/sin of the rotary angles pos * theta^(-2k/head_dim), k < head_dim/2, in fp64."""
    k = np.arange(head_dim // 2, dtype=F64)
    inv_freq = np.power(F64(theta), -2.0 * k / head_dim)
    ang = np.asarray(pos, F64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x, pos, theta):
    """Rotary embedding on x[n, H, hd] at positions pos[n].

    Pairing is (k, k + hd/2) ("rotate half"): the first half becomes
    x1 cos - x2 sin and the second half x2 cos + x1 sin.
    """
    x = np.asarray(x, F64)
    hd = x.shape[-1]
    c, s = rope_cos_sin(pos, hd, theta)
    c = c[:, None, :]
    s = s[:, None, :]
    x1, x2 = x[..., : hd // 2], x[..., hd // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    """GELU with the tanh approximation (GPT-2's MLP activation):
    0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    x = np.asarray(x, F64)
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def gelu_erf(x):
    erf = np.vectorize(math.erf, otypes=[F64])
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def softmax_rows(scores):
    m = np.max(scores, axis=-1, keepdims=True)
    e = np.exp(scores - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def as64(w):
    """Convert a weight dict tree to float64 arrays."""
    if isinstance(w, dict):
        return {k: as64(v) for k, v in w.items()}
    if isinstance(w, list):
        return [as64(v) for v in w]
    return np.asarray(w, F64)


# ---------------------------------------------------------------------------
# The exit policy (Section 4.1, Eq. 7-8; local variant Appendix H.3).
# ---------------------------------------------------------------------------

def cosine(h, ref):
    """Row-wise <h, ref> / (|h| |ref|) in fp64; NaN where either norm is 0.

    For the global metric ref is the inertia sum; Eq. 8 compares the unit
    vectors, which is this cosine.  For the local metric ref is h_{i-1}.
    """
    h = np.asarray(h, F64)
    ref = np.asarray(ref, F64)
    s_hh = np.einsum("nd,nd->n", h, h)
    s_rr = np.einsum("nd,nd->n", ref, ref)
    s_hr = np.einsum("nd,nd->n", h, ref)
    den = np.sqrt(s_hh) * np.sqrt(s_rr)
    out = np.full(h.shape[0], np.nan)
    ok = den > 0
    out[ok] = s_hr[ok] / den[ok]
    return out


def similarity(metric, h, inertia, h_prev):
    """The similarity the exit test compares with delta: the global cosine
    (with the inertia), the local one (with h_{i-1}), or for "both" the
    smaller of the two, so that sim >= delta exactly when both pass (NaN if
    either is undefined)."""
    if metric == GLOBAL:
        return cosine(h, inertia)
    if metric == LOCAL:
        return cosine(h, h_prev)
    if metric == BOTH:
        return np.minimum(cosine(h, inertia), cosine(h, h_prev))   # NaN propagates
    raise ValueError(metric)


def exit_decision(sim, layer, n_layers, delta, min_exit_layer):
    """Eq. 8: exit iff sim >= delta, tested only for min_exit_layer <= layer <= N-1.

    NaN (undefined cosine) never exits.  delta = +inf never fires.
    """
    sim = np.asarray(sim, F64)
    if not (min_exit_layer <= layer <= n_layers - 1):
        return np.zeros(sim.shape, bool)
    with np.errstate(invalid="ignore"):
        return sim >= delta


def inertia_update(inertia, h):
    """Eq. 7: add the unit-normalised current state to the running sum.

    A zero row adds nothing (its direction is undefined)."""
    h = np.asarray(h, F64)
    nrm = np.sqrt(np.einsum("nd,nd->n", h, h))
    add = np.zeros_like(h)
    ok = nrm > 0
    add[ok] = h[ok] / nrm[ok, None]
    return np.asarray(inertia, F64) + add


def compact(flags, active):
    """Appendix I: split the active index list by the exit flags.

    Returns (still_active, exited), each in the order of `active` (ascending
    when `active` is ascending)."""
    still = [int(a) for a, f in zip(active, flags) if not f]
    gone = [int(a) for a, f in zip(active, flags) if f]
    return np.array(still, np.int64), np.array(gone, np.int64)


# ---------------------------------------------------------------------------
# Decoupled KV generation (Section 4, Eq. 6; Section 4.3, Eq. 9).
# ---------------------------------------------------------------------------

def attn_input_norm(layer_w, shape, x):
    """The layer's pre-attention norm: RMSNorm (llama family) or LayerNorm
    with bias (gpt2 family)."""
    if shape.family == GPT2:
        return layer_norm(x, layer_w["ln1_g"], layer_w["ln1_b"], shape.ln_eps)
    return rms_norm(x, layer_w["attn_norm"], shape.rms_eps)


def _proj(u, layer_w, w, b, shape):
    y = u @ layer_w[w].T
    if shape.family == GPT2:
        y = y + layer_w[b]
    return y.reshape(u.shape[0], shape.n_heads, shape.head_dim)


def layer_kv(layer_w, x, pos, shape):
    """Layer r's own key/value path applied to input states x[n, D], as
    [n, H, hd]: llama K = RoPE(RMSNorm_r(x) Wk_r^T, pos), V = RMSNorm_r(x) Wv_r^T;
    gpt2 K = LN1_r(x) Wk_r^T + bk_r, V = LN1_r(x) Wv_r^T + bv_r (positions
    enter through the embedding, not the keys)."""
    u = attn_input_norm(layer_w, shape, x)
    k = _proj(u, layer_w, "wk", "bk", shape)
    v = _proj(u, layer_w, "wv", "bv", shape)
    if shape.family == GPT2:
        return k, v
    return apply_rope(k, pos, shape.rope_theta), v


def kv_generate(weights, shape, s_map, exit_layer, pos):
    """Eq. 9 for a set of exited tokens: for every skipped layer r > i*_j,
    s^{kv}_{r,j} = s~_j W_r^{kv}, with W_r^{kv} = [Wk_r | Wv_r] applied after
    layer r's pre-attention norm and with RoPE on the key half.

    s_map [n, D], exit_layer [n] (1-based i*), pos [n].
    Returns {r: (token_idx, K [m, H, hd], V [m, H, hd])} for r = 1..N, where
    token_idx lists the tokens with i* < r.  Layers are independent of each
    other (Eq. 6), so each is computed on its own.
    """
    s_map = np.asarray(s_map, F64)
    exit_layer = np.asarray(exit_layer)
    pos = np.asarray(pos)
    out = {}
    for r in range(1, shape.n_layers + 1):
        idx = np.nonzero(exit_layer < r)[0]
        if idx.size == 0:
            continue
        k, v = layer_kv(weights["layers"][r - 1], s_map[idx], pos[idx], shape)
        out[r] = (idx, k, v)
    return out


# ---------------------------------------------------------------------------
# Attention over a key/value cache that mixes computed and generated entries
# (Section 3, Eq. 5; Section 4.3).
# ---------------------------------------------------------------------------

def attend(q, k_cache, v_cache, slot_base, pos, key_len=None, causal=True, key_mask=None):
    """Softmax attention of queries q[n, H, hd] over cache rows.

    Query j reads cache slots slot_base[j] + t for t in [0, pos[j]] when
    causal, else t in [0, key_len[j]); key_mask (bool [n, L]) optionally
    removes keys.  Cache entries must all be defined (NaN-poisoned
    unwritten slots propagate and are caught by the tests).
    """
    n, H, hd = q.shape
    out = np.empty((n, H, hd), F64)
    scale = 1.0 / math.sqrt(hd)
    for j in range(n):
        L = int(pos[j]) + 1 if causal else int(key_len[j])
        sl = slice(int(slot_base[j]), int(slot_base[j]) + L)
        K = k_cache[sl]   # [L, H, hd]
        V = v_cache[sl]
        s = np.einsum("hd,lhd->hl", q[j], K) * scale
        if key_mask is not None:
            s = np.where(key_mask[j][None, :L], s, -np.inf)
        p = softmax_rows(s)
        out[j] = np.einsum("hl,lhd->hd", p, V)
    return out


# ---------------------------------------------------------------------------
# Generative forward with token-level exit (Section 4, Appendix I).
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class ExitConfig:
    delta: float = math.inf        # Eq. 8 threshold; +inf never fires
    min_exit_layer: int = 1
    metric: str = GLOBAL
    prompt_level: bool = False     # all-at-once variant (Appendix H.2)


@dataclasses.dataclass
class KVCache:
    """Per-layer key/value cache [N, B * s_max, H, hd]; slot of (b, p) = b * s_max + p."""
    k: np.ndarray
    v: np.ndarray
    s_max: int

    @classmethod
    def empty(cls, shape, batch, s_max):
        dims = (shape.n_layers, batch * s_max, shape.n_heads, shape.head_dim)
        return cls(np.full(dims, np.nan), np.full(dims, np.nan), s_max)


@dataclasses.dataclass
class TokenPassResult:
    h_final: np.ndarray        # [n, D]: h_{i*} for exited tokens, h_N otherwise
    exit_layer: np.ndarray     # [n], 1-based; N means never exited
    logits: np.ndarray         # [n, V]
    sims: np.ndarray           # [N, n] cosine at each layer (NaN where not tested/inactive)
    active_counts: list        # active rows entering each layer 1..N
    hidden: list               # hidden[i] = [n, D] states after layer i (frozen rows for exited)
    inertia: np.ndarray        # [n, D] inertia after the last test (global metric)


def layer_q(layer_w, shape, h_in, pos):
    """Layer i's queries of input states h_in[n, D], [n, H, hd]: llama
    RoPE(RMSNorm_i(h_in) Wq_i^T); gpt2 LN1_i(h_in) Wq_i^T + bq_i."""
    q = _proj(attn_input_norm(layer_w, shape, h_in), layer_w, "wq", "bq", shape)
    if shape.family == GPT2:
        return q
    return apply_rope(q, pos, shape.rope_theta)


def layer_out(layer_w, shape, h_in, o):
    """The rest of a regular layer after attention: output projection and
    residual, then the FFN on its normalised input and the second residual.
    llama: RMSNorm and SwiGLU; gpt2: LayerNorm, GELU (tanh form), biases.
    h_in [n, D] = h_{i-1}, o [n, H, hd] = attention output."""
    n = h_in.shape[0]
    h1 = np.asarray(h_in, F64) + np.asarray(o, F64).reshape(n, -1) @ layer_w["wo"].T
    if shape.family == GPT2:
        h1 = h1 + layer_w["bo"]
        u2 = layer_norm(h1, layer_w["ln2_g"], layer_w["ln2_b"], shape.ln_eps)
        ff = gelu_tanh(u2 @ layer_w["w_fc"].T + layer_w["b_fc"]) @ layer_w["w_proj"].T
        return h1 + ff + layer_w["b_proj"]
    u2 = rms_norm(h1, layer_w["ffn_norm"], shape.rms_eps)
    ff = (silu(u2 @ layer_w["w_gate"].T) * (u2 @ layer_w["w_up"].T)) @ layer_w["w_down"].T
    return h1 + ff


def embed_rows(weights, shape, ids, pos):
    """h_0 of token rows: the token embedding, plus the learned position
    embedding for the gpt2 family."""
    h0 = np.asarray(weights["embed"], F64)[np.asarray(ids)]
    if shape.family == GPT2:
        h0 = h0 + np.asarray(weights["pos_embed"], F64)[np.asarray(pos)]
    return h0


def decoder_layer(layer_w, shape, h_in, pos, seq, cache, layer):
    """One regular decoder layer for the active rows (Appendix I, "Process 1").

    h_in [n, D] are the rows' states h_{i-1}; their own K/V are written to
    the cache first, then every row attends causally over its sequence."""
    q = layer_q(layer_w, shape, h_in, pos)
    k, v = layer_kv(layer_w, h_in, pos, shape)
    slots = seq * cache.s_max + pos
    cache.k[layer - 1][slots] = k
    cache.v[layer - 1][slots] = v
    o = attend(q, cache.k[layer - 1], cache.v[layer - 1], seq * cache.s_max, pos)
    return layer_out(layer_w, shape, h_in, o)


def lm_logits(weights, shape, h_final):
    """Final norm and LM head of final states h_final[n, D] (an exited
    token's final state is its mapped state, Fig. 1 caption): llama RMSNorm
    and an untied head; gpt2 LayerNorm and the token embedding as the head."""
    if shape.family == GPT2:
        u = layer_norm(h_final, weights["final_ln_g"], weights["final_ln_b"], shape.ln_eps)
        return u @ np.asarray(weights["embed"], F64).T
    return rms_norm(h_final, weights["final_norm"], shape.rms_eps) @ weights["lm_head"].T


def token_pass(weights, shape, h0, pos, seq, cache, cfg, force_layer=None, mapper=None):
    """Run a set of token rows through the N layers with token-level exit.

    This is the prefill of Appendix I when the rows are a whole prompt batch,
    and one generation step when the rows are the newly sampled tokens (each
    at the end of its sequence).  Per layer i:
      1. the active rows run the regular layer (own K/V into cache[i]);
      2. the exit test of Eq. 8 (global: against the inertia of Eq. 7, then
         the inertia update; local: against h_{i-1});
      3. the active list is split into still-active and exited rows;
      4. the exited rows' K/V for every layer r > i are generated (Eq. 9).
    force_layer (optional int [n]): a value f > 0 replaces the policy for that
    row by "exit exactly at layer f" (f >= N: never); 0 keeps the policy.
    mapper (optional): s~ = mapper(h_i, h_{i-1}, inertia before layer i's
    update) for the rows exiting at layer i (Section 4.2); s~ replaces h_i as
    the exited row's state, so its generated K/V and its final state use it.
    None is the identity mapper.
    """
    N, D = shape.n_layers, shape.d_model
    h0 = np.asarray(h0, F64)
    n = h0.shape[0]
    pos = np.asarray(pos, np.int64)
    seq = np.asarray(seq, np.int64)
    h = h0.copy()
    inertia = np.zeros((n, D))
    exit_layer = np.full(n, N, np.int64)
    active = np.arange(n)
    sims = np.full((N, n), np.nan)
    counts, hidden = [], []
    for i in range(1, N + 1):
        counts.append(int(active.size))
        h_prev = h.copy()
        if active.size:
            h[active] = decoder_layer(weights["layers"][i - 1], shape, h_prev[active],
                                      pos[active], seq[active], cache, i)
        sim = (similarity(cfg.metric, h[active], inertia[active], h_prev[active])
               if active.size else np.zeros(0))
        sims[i - 1, active] = sim
        flags = exit_decision(sim, i, N, cfg.delta, cfg.min_exit_layer)
        if force_layer is not None:
            f = np.asarray(force_layer)[active]
            forced = f > 0
            flags = np.where(forced, (f == i) & (i <= N - 1), flags)
        if cfg.prompt_level and active.size:
            # Appendix H.2: each prompt's last token (its active row of
            # largest position) decides for all of the prompt's tokens
            sa, pa = seq[active], pos[active]
            for b in np.unique(sa):
                members = np.nonzero(sa == b)[0]
                flags[members] = flags[members[np.argmax(pa[members])]]
        inertia_pre = inertia.copy() if mapper is not None else None
        if cfg.metric != LOCAL and active.size:
            inertia[active] = inertia_update(inertia[active], h[active])
        active, exited = compact(flags, active)
        exit_layer[exited] = i
        if mapper is not None and exited.size and i < N:
            h[exited] = mapper(h[exited], h_prev[exited], inertia_pre[exited])
        if exited.size and i < N:
            gen = kv_generate(weights, shape, h[exited], exit_layer[exited], pos[exited])
            for r, (idx, k, v) in gen.items():
                slots = seq[exited[idx]] * cache.s_max + pos[exited[idx]]
                cache.k[r - 1][slots] = k
                cache.v[r - 1][slots] = v
        hidden.append(h.copy())
    return TokenPassResult(h, exit_layer, lm_logits(weights, shape, h), sims, counts, hidden,
                           inertia)


def prefill(weights, shape, ids, cfg, s_max=None, force_layer=None, mapper=None):
    """Prefill of a [B, T] prompt batch; rows are j = b*T + p (Appendix I's
    [4N, D_h] flattening).  Returns (TokenPassResult, KVCache)."""
    ids = np.asarray(ids)
    B, T = ids.shape
    s_max = T if s_max is None else s_max
    cache = KVCache.empty(shape, B, s_max)
    pos = np.tile(np.arange(T), B)
    seq = np.repeat(np.arange(B), T)
    h0 = embed_rows(weights, shape, ids.reshape(-1), pos)
    res = token_pass(weights, shape, h0, pos, seq, cache, cfg,
                     None if force_layer is None else np.asarray(force_layer).reshape(-1),
                     mapper=mapper)
    return res, cache


def greedy(logits):
    """Greedy choice with ties going to the lowest token id."""
    return np.argmax(np.asarray(logits), axis=-1)


def decode_step(weights, shape, cache, ids, pos, cfg, force_layer=None, mapper=None):
    """One generation step (Appendix I, generation phase): token ids[b] sits
    at position pos[b] of sequence b; inertia starts empty for the new token."""
    ids = np.asarray(ids)
    B = ids.shape[0]
    h0 = embed_rows(weights, shape, ids, pos)
    return token_pass(weights, shape, h0, np.asarray(pos), np.arange(B), cache, cfg, force_layer,
                      mapper=mapper)


def generate(weights, shape, ids, n_steps, cfg, force_layer=None, mapper=None):
    """Prefill of ids [B, T] then n_steps greedy generation steps.
    Returns (prefill result, list of step results, generated ids [B, n_steps], cache)."""
    B, T = np.asarray(ids).shape
    res, cache = prefill(weights, shape, ids, cfg, s_max=T + n_steps, force_layer=force_layer,
                         mapper=mapper)
    last = res.logits.reshape(B, T, -1)[:, -1]
    nxt = greedy(last)
    steps, out = [], []
    for s in range(n_steps):
        out.append(nxt)
        st = decode_step(weights, shape, cache, nxt, np.full(B, T + s), cfg, mapper=mapper)
        steps.append(st)
        nxt = greedy(st.logits)
    return res, steps, np.stack(out, axis=1) if out else np.zeros((B, 0), np.int64), cache


def full_depth_logits(weights, shape, ids):
    """The base model without exits (delta = +inf) -- the reference point of
    every compute-reduction figure in the paper."""
    res, _ = prefill(weights, shape, ids, ExitConfig(delta=math.inf))
    return res.logits


# ---------------------------------------------------------------------------
# Classification mode (Section 4.3, "downstream tasks"): post-norm encoder,
# computation stops at the exit layer, no KV generation.
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class ClassifyResult:
    logits: np.ndarray       # [B, n_classes] from the [CLS] state at its exit
    exit_layer: np.ndarray   # [B*T]
    cls_exit_layer: np.ndarray
    h_final: np.ndarray
    sims: np.ndarray
    active_counts: list


def encoder_layer(lw, shape, x, seq):
    """One post-norm encoder layer over the live (still active) tokens x[m, D]
    of their sequences seq[m]: bidirectional attention of each token over the
    live tokens of its own sequence, LayerNorm after each residual, GELU FFN."""
    return encoder_ffn_block(lw, shape, encoder_attention_block(lw, shape, x, seq))


def encoder_qkv(lw, shape, x):
    """Queries, keys and values (with biases) of encoder states x[m, D], [m, H, hd] each."""
    x = np.asarray(x, F64)
    m, H, hd = x.shape[0], shape.n_heads, shape.head_dim
    return tuple((x @ lw[w].T + lw[b]).reshape(m, H, hd)
                 for w, b in (("wq", "bq"), ("wk", "bk"), ("wv", "bv")))


def encoder_attend(q, kk, vv, seq):
    """Bidirectional attention of each live token over the live tokens of its
    own sequence (rows with the same seq), per head."""
    q, kk, vv = (np.asarray(t, F64) for t in (q, kk, vv))
    scale = 1.0 / math.sqrt(q.shape[-1])
    o = np.empty(q.shape)
    seq = np.asarray(seq)
    for b in np.unique(seq):
        rows = np.nonzero(seq == b)[0]           # live tokens of sequence b
        s = np.einsum("qhd,khd->hqk", q[rows], kk[rows]) * scale
        o[rows] = np.einsum("hqk,khd->qhd", softmax_rows(s), vv[rows])
    return o


def encoder_attention_out(lw, shape, x, o):
    """LayerNorm_1(x + o Wo^T + bo): the attention sub-layer's output from its
    input x[m, D] and the attention output o[m, H, hd]."""
    x = np.asarray(x, F64)
    return layer_norm(x + np.asarray(o, F64).reshape(x.shape[0], -1) @ lw["wo"].T + lw["bo"],
                      lw["ln1_g"], lw["ln1_b"], shape.ln_eps)


def encoder_attention_block(lw, shape, x, seq):
    """The attention sub-layer of a post-norm encoder layer:
    LayerNorm_1(x + Attention(x) Wo^T + bo) for the live tokens x[m, D]."""
    q, kk, vv = encoder_qkv(lw, shape, x)
    return encoder_attention_out(lw, shape, x, encoder_attend(q, kk, vv, seq))


def encoder_ffn_block(lw, shape, h1):
    """The FFN sub-layer of a post-norm encoder layer:
    LayerNorm_2(h1 + GELU(h1 W_in^T + b_in) W_out^T + b_out)."""
    h1 = np.asarray(h1, F64)
    ff = gelu_erf(h1 @ lw["w_in"].T + lw["b_in"]) @ lw["w_out"].T + lw["b_out"]
    return layer_norm(h1 + ff, lw["ln2_g"], lw["ln2_b"], shape.ln_eps)


def classify_logits(weights, cls_states):
    """The linear head on [CLS] states (Section 4.3: the mapped state feeds the classifier)."""
    return (np.asarray(cls_states, F64) @ np.asarray(weights["cls_w"], F64).T
            + np.asarray(weights["cls_b"], F64))


def cls_stop(flags, active, seq_len):
    """Early stop of a classification sequence (Section 4.3: the computation
    ends once the state that feeds the classifier has exited): a row leaves
    at the layer where its sequence's [CLS] row (row b * seq_len, position 0)
    exits, or at once if that row is no longer active.  flags [n] over the
    active rows (ascending)."""
    act = np.asarray(active)
    flags = np.asarray(flags, bool)
    if act.size == 0:
        return flags
    cls = (act // seq_len) * seq_len
    k = np.minimum(np.searchsorted(act, cls), act.size - 1)
    present = act[k] == cls
    return flags | ~present | flags[k]


def classify(weights, shape, ids, cfg, force_layer=None, stop_at_cls=True):
    """Token-level exit in an encoder classifier.

    Readings: exited tokens stop entirely (no KV generation) and leave the
    key set of later layers; a sequence's output is the [CLS] (position 0)
    state at its exit, fed to the linear head.  Tokens of a sequence whose
    [CLS] has exited no longer influence the output, so with stop_at_cls
    they leave at that layer too (cls_stop); the logits are the same either
    way."""
    ids = np.asarray(ids)
    B, T = ids.shape
    N, D, H, hd = shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim
    n = B * T
    pos = np.tile(np.arange(T), B)
    seq = np.repeat(np.arange(B), T)
    x = (np.asarray(weights["word_embed"], F64)[ids.reshape(-1)]
         + np.asarray(weights["pos_embed"], F64)[pos] + np.asarray(weights["type_embed"], F64))
    h = layer_norm(x, weights["embed_ln_g"], weights["embed_ln_b"], shape.ln_eps)
    inertia = np.zeros((n, D))
    exit_layer = np.full(n, N, np.int64)
    live = np.ones(n, bool)
    active = np.arange(n)
    sims = np.full((N, n), np.nan)
    counts = []
    for i in range(1, N + 1):
        counts.append(int(active.size))
        lw = weights["layers"][i - 1]
        h_prev = h.copy()
        if active.size:
            h[active] = encoder_layer(lw, shape, h_prev[active], seq[active])
        sim = (similarity(cfg.metric, h[active], inertia[active], h_prev[active])
               if active.size else np.zeros(0))
        sims[i - 1, active] = sim
        flags = exit_decision(sim, i, N, cfg.delta, cfg.min_exit_layer)
        if force_layer is not None:
            f = np.asarray(force_layer).reshape(-1)[active]
            forced = f > 0
            flags = np.where(forced, (f == i) & (i <= N - 1), flags)
        if stop_at_cls:
            flags = cls_stop(flags, active, T)
        if cfg.metric != LOCAL and active.size:
            inertia[active] = inertia_update(inertia[active], h[active])
        active, exited = compact(flags, active)
        exit_layer[exited] = i
        live[exited] = False
    cls_rows = np.arange(B) * T
    return ClassifyResult(classify_logits(weights, h[cls_rows]), exit_layer, exit_layer[cls_rows],
                          h, sims, counts)
