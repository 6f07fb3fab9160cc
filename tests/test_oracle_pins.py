"""Pins of the CPU oracle against things other than itself.

Each test ties an oracle function to a value the paper prints, a closed
form, an independent library implementation (transformers' Llama/BERT in
fp64, torch functional ops) or a brute-force recomputation.  A plausible
mistake in the oracle (a dropped term, a wrong sign or index, a transposed
operand, a wrong layer) fails at least one of them; test_planted_mistakes
checks that claim for a few such mistakes.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import accounting as acc
from oracle import adept_oracle as O
from oracle import brute_force as BF
from tests import hf_models

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SMALL = ai.DecoderShape(n_layers=4, d_model=64, n_heads=4, head_dim=16, d_ff=128, vocab=97)


@pytest.fixture(scope="module")
def small():
    w = O.as64(ai.decoder_weights(SMALL, seed=11))
    ids = ai.token_ids(12, SMALL.vocab, 2, 12)
    return w, ids


def _quantile_delta(w, ids, metric, layer, q):
    """A threshold at quantile q of the layer's similarities (so it fires for
    part of the tokens)."""
    res, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf, metric=metric))
    s = res.sims[layer - 1]
    return float(np.quantile(s[np.isfinite(s)], q))


# --------------------------------------------------------------------------
# base-model building blocks vs library implementations / closed forms
# --------------------------------------------------------------------------

def test_rms_norm_matches_torch():
    x = np.random.default_rng(0).standard_normal((5, 33))
    g = np.random.default_rng(1).standard_normal(33)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-6)
    np.testing.assert_allclose(O.rms_norm(x, g, 1e-6), ref.numpy(), rtol=1e-13, atol=0)


def test_layer_norm_matches_torch():
    x = np.random.default_rng(0).standard_normal((5, 33)) * 3 + 1
    g = np.random.default_rng(1).standard_normal(33)
    b = np.random.default_rng(2).standard_normal(33)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (33,), torch.from_numpy(g),
                                         torch.from_numpy(b), eps=1e-12)
    np.testing.assert_allclose(O.layer_norm(x, g, b, 1e-12), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_gelu_and_silu_match_torch():
    x = np.linspace(-6, 6, 101)
    np.testing.assert_allclose(O.gelu_erf(x), torch.nn.functional.gelu(torch.from_numpy(x)).numpy(),
                               rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(O.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-14, atol=1e-15)


def test_rope_properties():
    rng = np.random.default_rng(3)
    H, hd = 3, 16
    x = rng.standard_normal((4, H, hd))
    # position 0 is the identity
    np.testing.assert_allclose(O.apply_rope(x, np.zeros(4), 10000.0), x, rtol=0, atol=0)
    # every (k, k + hd/2) pair keeps its length
    pos = np.array([1, 7, 100, 4095])
    y = O.apply_rope(x, pos, 10000.0)
    n_x = x[..., :8] ** 2 + x[..., 8:] ** 2
    n_y = y[..., :8] ** 2 + y[..., 8:] ** 2
    np.testing.assert_allclose(n_y, n_x, rtol=1e-13)
    # it is multiplication of z_k = x_k + i x_{k+hd/2} by exp(i pos theta^(-2k/hd))
    z = x[..., :8] + 1j * x[..., 8:]
    rot = np.exp(1j * pos[:, None, None] * 10000.0 ** (-np.arange(8) * 2 / hd))
    zr = z * rot
    np.testing.assert_allclose(y[..., :8], zr.real, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[..., 8:], zr.imag, rtol=1e-12, atol=1e-12)
    # scores depend only on the position difference
    q, k = rng.standard_normal((1, 1, hd)), rng.standard_normal((1, 1, hd))
    s1 = np.sum(O.apply_rope(q, [9], 1e4) * O.apply_rope(k, [4], 1e4))
    s2 = np.sum(O.apply_rope(q, [109], 1e4) * O.apply_rope(k, [104], 1e4))
    assert abs(s1 - s2) < 1e-12


def test_attention_matches_sdpa():
    rng = np.random.default_rng(5)
    T, H, hd = 9, 2, 8
    q = rng.standard_normal((T, H, hd))
    k = rng.standard_normal((T, H, hd))
    v = rng.standard_normal((T, H, hd))
    out = O.attend(q, k, v, np.zeros(T, int), np.arange(T))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1), torch.from_numpy(k).transpose(0, 1),
        torch.from_numpy(v).transpose(0, 1), is_causal=True).transpose(0, 1)
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------------------
# the exit policy (Section 4.1 Eq. 7-8, Appendix H.3)
# --------------------------------------------------------------------------

def test_cosine_closed_forms():
    rng = np.random.default_rng(7)
    a = rng.standard_normal(40)
    b = rng.standard_normal(40)
    b_perp = b - a * (a @ b) / (a @ a)
    rows = np.stack([a, a, a, a, np.zeros(40), a])
    refs = np.stack([3.5 * a, b_perp, -2 * a, b, a, np.zeros(40)])
    s = O.cosine(rows, refs)
    assert abs(s[0] - 1) < 1e-15 and abs(s[1]) < 1e-15 and abs(s[2] + 1) < 1e-15
    ref = torch.nn.functional.cosine_similarity(torch.from_numpy(a), torch.from_numpy(b), dim=0)
    assert abs(s[3] - float(ref)) < 1e-14
    assert np.isnan(s[4]) and np.isnan(s[5])


def test_both_metric_is_and_of_global_and_local():
    """The combined metric (a reading: Appendix H.3 does not define it) exits
    only where both cosines pass; built from rows with known cosines."""
    rng = np.random.default_rng(11)
    a = rng.standard_normal(32)
    b = rng.standard_normal(32)
    b_perp = b - a * (a @ b) / (a @ a)
    z = np.zeros(32)
    #              global passes, local fails | local passes, global fails | both | none | NaN
    h = np.stack([a, a, a, a, a])
    inertia = np.stack([2 * a, b_perp, 5 * a, -a, z])
    prev = np.stack([b_perp, 0.5 * a, 3 * a, b_perp, a])
    sim = O.similarity(O.BOTH, h, inertia, prev)
    np.testing.assert_allclose(sim[:4], [0.0, 0.0, 1.0, -1.0], atol=1e-15)
    assert np.isnan(sim[4])
    assert O.exit_decision(sim, 2, 4, 0.5, 1).tolist() == [False, False, True, False, False]
    # the single metrics on the same rows
    assert O.exit_decision(O.similarity(O.GLOBAL, h, inertia, prev), 2, 4, 0.5, 1).tolist() == \
        [True, False, True, False, False]
    assert O.exit_decision(O.similarity(O.LOCAL, h, inertia, prev), 2, 4, 0.5, 1).tolist() == \
        [False, True, True, False, True]


def test_exit_decision_window_and_special_thresholds():
    s = np.array([0.5, 0.97, np.nan, 1.0])
    assert O.exit_decision(s, 2, 4, 0.95, 1).tolist() == [False, True, False, True]
    assert not O.exit_decision(s, 4, 4, 0.95, 1).any()          # never at the last layer
    assert not O.exit_decision(s, 1, 4, 0.95, 2).any()          # below the minimum layer
    assert not O.exit_decision(s, 2, 4, math.inf, 1).any()      # +inf never fires
    assert O.exit_decision(s, 2, 4, -1.0, 1).tolist() == [True, True, False, True]


def test_inertia_is_sum_of_unit_states(small):
    """Eq. 7: after layer i the inertia equals the sum of h_d/|h_d|, d <= i,
    recomputed from the recorded per-layer states."""
    w, ids = small
    res, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf, metric=O.GLOBAL))
    acc_ = sum(h / np.linalg.norm(h, axis=1, keepdims=True) for h in res.hidden)
    np.testing.assert_allclose(res.inertia, acc_, rtol=1e-13, atol=1e-13)
    # and the sim at layer i is cos(h_i, sum_{d<i} h_d/|h_d|)
    i = 3
    ref = sum(h / np.linalg.norm(h, axis=1, keepdims=True) for h in res.hidden[: i - 1])
    h = res.hidden[i - 1]
    c = np.sum(h * ref, 1) / np.linalg.norm(h, axis=1) / np.linalg.norm(ref, axis=1)
    np.testing.assert_allclose(res.sims[i - 1], c, rtol=1e-13)


def test_global_equals_local_at_layer_two(small):
    """With one previous layer the inertia is the unit vector of h_1, so both metrics agree."""
    w, ids = small
    g, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf, metric=O.GLOBAL))
    l, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf, metric=O.LOCAL))
    np.testing.assert_allclose(g.sims[1], l.sims[1], rtol=1e-13)
    assert np.isnan(g.sims[0]).all()          # empty inertia at layer 1
    assert np.isfinite(l.sims[0]).all()


def test_compact_is_flatnonzero():
    rng = np.random.default_rng(9)
    active = np.sort(rng.choice(1000, 300, replace=False))
    flags = rng.random(300) < 0.3
    still, gone = O.compact(flags, active)
    np.testing.assert_array_equal(still, active[np.flatnonzero(~flags)])
    np.testing.assert_array_equal(gone, active[np.flatnonzero(flags)])
    e1, e2 = O.compact(np.zeros(0, bool), np.zeros(0, int))
    assert e1.size == 0 and e2.size == 0


def test_appendix_i_worked_example(small):
    """Appendix I: in "I am a person", <am> exits after layer 1 and <a> after
    layer 2, so the active tensor shrinks 4 -> 3 -> 2 rows."""
    ex = json.load(open(os.path.join(GOLDEN, "appendix_i_worked_example.json")))
    w, _ = small
    toks = ex["prompt_tokens"]
    ids = np.array([[3, 17, 29, 41]])
    force = np.zeros((1, 4), int)
    for t, layer in ex["forced_exit_layer"].items():
        force[0, toks.index(t)] = layer
    res, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf), force_layer=force)
    for layer, n in ex["active_rows_entering_layer"].items():
        assert res.active_counts[int(layer) - 1] == n
    assert res.exit_layer.tolist() == [4, 1, 2, 4]
    # a batch of n prompts is the [4n, D] flattening: the same counts times n
    res3, _ = O.prefill(w, SMALL, np.repeat(ids, 3, 0), O.ExitConfig(delta=math.inf),
                        force_layer=np.repeat(force, 3, 0))
    assert res3.active_counts[:3] == [12, 9, 6]
    # generation example: <with> exits after layer 2, <happiness> after layer 3
    gen = ex["generation_example"]
    _, cache = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf), s_max=6)
    for step, tok in enumerate(gen["tokens"]):
        st = O.decode_step(w, SMALL, cache, np.array([50 + step]), np.array([4 + step]),
                           O.ExitConfig(delta=math.inf),
                           force_layer=np.array([gen["exit_layer"][tok]]))
        assert st.exit_layer.tolist() == [gen["exit_layer"][tok]]
        assert st.active_counts == [1 if i in gen["layers_executed"][tok] else 0
                                    for i in range(1, SMALL.n_layers + 1)]


# --------------------------------------------------------------------------
# the whole forward vs transformers (full depth, truncated depth) and vs the
# token-at-a-time brute force
# --------------------------------------------------------------------------

def test_full_depth_matches_transformers_llama(small):
    """delta = +inf (never exits) is the plain base model: logits and the
    K/V cache equal transformers' LlamaForCausalLM in fp64.  (transformers
    forms the RMSNorm statistics and the rotary angles in fp32 even in an
    fp64 model, so agreement is to about 1e-7, far below what a wrong sign,
    index or operand would give.)"""
    w, ids = small
    res, cache = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf))
    m = hf_models.llama(SMALL, w)
    with torch.no_grad():
        out = m(torch.from_numpy(ids.astype(np.int64)), use_cache=True)
    B, T = ids.shape
    np.testing.assert_allclose(res.logits.reshape(B, T, -1), out.logits.numpy(), rtol=0, atol=2e-7)
    for i in range(SMALL.n_layers):
        hk = out.past_key_values.layers[i].keys.numpy()      # [B, H, T, hd]
        hv = out.past_key_values.layers[i].values.numpy()
        ok = cache.k[i].reshape(B, T, SMALL.n_heads, SMALL.head_dim).transpose(0, 2, 1, 3)
        ov = cache.v[i].reshape(B, T, SMALL.n_heads, SMALL.head_dim).transpose(0, 2, 1, 3)
        np.testing.assert_allclose(ok, hk, rtol=0, atol=1e-7)
        np.testing.assert_allclose(ov, hv, rtol=0, atol=1e-7)
    assert (res.exit_layer == SMALL.n_layers).all()


@pytest.mark.parametrize("k", [1, 2, 3])
def test_exit_everything_at_k_is_truncated_model(small, k):
    """delta = -1, local metric, minimum exit layer k: every token exits at k.
    Logits equal the k-layer truncated model's (transformers), and the
    generated K/V of every layer r > k equal transformers' own layer-r key and
    value path applied to h_k (Eq. 9 with the identity mapper)."""
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    w, ids = small
    res, cache = O.prefill(w, SMALL, ids, O.ExitConfig(delta=-1.0, min_exit_layer=k,
                                                       metric=O.LOCAL))
    assert (res.exit_layer == k).all()
    B, T = ids.shape
    m = hf_models.llama(SMALL, w, n_layers=k)
    tid = torch.from_numpy(ids.astype(np.int64))
    with torch.no_grad():
        out = m(tid, output_hidden_states=True)
    np.testing.assert_allclose(res.logits.reshape(B, T, -1), out.logits.numpy(), rtol=0, atol=2e-7)
    full = hf_models.llama(SMALL, w)
    posid = torch.arange(T)[None, :].repeat(B, 1)
    with torch.no_grad():
        # the full model's input to layer k+1 is h_k (the last entry of the
        # truncated model's tuple is taken after the final norm)
        hk = full(tid, output_hidden_states=True).hidden_states[k]
        cos, sin = full.model.rotary_emb(hk, posid)
        for r in range(k + 1, SMALL.n_layers + 1):
            L = full.model.layers[r - 1]
            u = L.input_layernorm(hk)
            kk = L.self_attn.k_proj(u).view(B, T, SMALL.n_heads, SMALL.head_dim).transpose(1, 2)
            vv = L.self_attn.v_proj(u).view(B, T, SMALL.n_heads, SMALL.head_dim).transpose(1, 2)
            kk, _ = apply_rotary_pos_emb(kk, kk, cos, sin)
            ok = cache.k[r - 1].reshape(B, T, SMALL.n_heads, SMALL.head_dim).transpose(0, 2, 1, 3)
            ov = cache.v[r - 1].reshape(B, T, SMALL.n_heads, SMALL.head_dim).transpose(0, 2, 1, 3)
            np.testing.assert_allclose(ok, kk.numpy(), rtol=0, atol=1e-7)
            np.testing.assert_allclose(ov, vv.numpy(), rtol=0, atol=1e-7)


CASES = [("global", 2, 0.5, False), ("global", 3, 0.3, False), ("local", 1, 0.6, False),
         ("local", 2, 0.5, False), ("global", 2, 0.5, True), ("both", 2, 0.4, False),
         ("both", 3, 0.3, False)]


@pytest.mark.parametrize("metric,layer,q,forced", CASES)
def test_batched_prefill_equals_token_at_a_time(small, metric, layer, q, forced):
    """The batched prefill with compaction and decoupled KV generation gives
    the same logits, exit layers and caches as processing each token alone
    in order (causality makes the two equal)."""
    w, ids = small
    delta = _quantile_delta(w, ids, metric, layer, q)
    cfg = O.ExitConfig(delta=delta, metric=metric)
    force = None
    if forced:
        force = np.random.default_rng(4).integers(0, SMALL.n_layers + 1, size=ids.shape)
    res, cache = O.prefill(w, SMALL, ids, cfg, force_layer=force)
    assert 0 < np.sum(res.exit_layer < SMALL.n_layers) < ids.size or forced
    bf = BF.brute_force_prefill(w, SMALL, ids, cfg, force_layer=force)
    B, T = ids.shape
    for b in range(B):
        np.testing.assert_array_equal(res.exit_layer[b * T:(b + 1) * T], bf[b]["exit_layer"])
        np.testing.assert_allclose(res.logits[b * T:(b + 1) * T], bf[b]["logits"], rtol=0,
                                   atol=1e-12)
        for r in range(SMALL.n_layers):
            np.testing.assert_allclose(cache.k[r][b * T:(b + 1) * T], np.stack(bf[b]["keys"][r]),
                                       rtol=0, atol=1e-12)
            np.testing.assert_allclose(cache.v[r][b * T:(b + 1) * T],
                                       np.stack(bf[b]["values"][r]), rtol=0, atol=1e-12)


@pytest.mark.parametrize("metric", ["global", "local"])
def test_all_at_once_follows_last_prompt_token(small, metric):
    """All-at-once variant (Appendix H.2): a prompt's tokens all run until the
    first layer at which the prompt's last token passes the test, and that
    token's path equals the no-exit run's up to there (every key it attends
    to is then still computed), so the exit layer of each prompt can be read
    off the no-exit similarities of its last token; each token's final state
    is its state after that layer in the no-exit run."""
    w, ids = small
    B, T = ids.shape
    N = SMALL.n_layers
    full, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf, metric=metric))
    last = np.arange(B) * T + T - 1
    s_last = full.sims[:, last]                       # [N, B]
    tested = s_last[: N - 1]
    distinct = 0
    for delta in np.quantile(tested[np.isfinite(tested)], [0.3, 0.5, 0.7, 0.9]):
        res, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=float(delta), metric=metric,
                                                       prompt_level=True))
        for b in range(B):
            fire = [i for i in range(1, N) if s_last[i - 1, b] >= delta]
            want = fire[0] if fire else N
            rows = np.arange(b * T, (b + 1) * T)
            assert (res.exit_layer[rows] == want).all(), (b, want, res.exit_layer[rows])
            np.testing.assert_allclose(res.h_final[rows], full.hidden[want - 1][rows], rtol=0,
                                       atol=1e-12)
        distinct += len(set(res.exit_layer.tolist())) > 1
    assert distinct > 0          # some threshold gives the prompts different exit layers
    # token-level exits differ: the variant is not the method
    tok, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=float(np.median(s_last[1:N - 1])),
                                                   metric=metric))
    assert len(set(tok.exit_layer[:T].tolist())) > 1


def test_generation_matches_transformers_greedy(small):
    """Full depth: prefill then greedy steps equal transformers' cached decoding."""
    w, ids = small
    n_steps = 5
    res, steps, gen, _ = O.generate(w, SMALL, ids, n_steps, O.ExitConfig(delta=math.inf))
    m = hf_models.llama(SMALL, w)
    B, T = ids.shape
    with torch.no_grad():
        out = m(torch.from_numpy(ids.astype(np.int64)), use_cache=True)
        pkv = out.past_key_values
        nxt = out.logits[:, -1].argmax(-1)
        for s in range(n_steps):
            assert nxt.tolist() == gen[:, s].tolist()
            o = m(nxt[:, None], past_key_values=pkv, use_cache=True,
                  position_ids=torch.full((B, 1), T + s))
            pkv = o.past_key_values
            np.testing.assert_allclose(steps[s].logits, o.logits[:, 0].numpy(), rtol=0, atol=2e-7)
            nxt = o.logits[:, 0].argmax(-1)


@pytest.mark.parametrize("metric", ["global", "local", "both"])
def test_generation_with_exits_equals_token_at_a_time(small, metric):
    """Generation steps with token-level exits (Appendix I, generation phase)
    equal the token-at-a-time recomputation over prompt + generated tokens."""
    w, ids = small
    delta = _quantile_delta(w, ids, metric, 2, 0.5)
    cfg = O.ExitConfig(delta=delta, metric=metric)
    res, steps, gen, _ = O.generate(w, SMALL, ids, 4, cfg)
    allids = np.concatenate([ids, gen], axis=1)
    bf = BF.brute_force_prefill(w, SMALL, allids, cfg)
    T = ids.shape[1]
    for b in range(ids.shape[0]):
        for s, st in enumerate(steps):
            assert st.exit_layer[b] == bf[b]["exit_layer"][T + s]
            np.testing.assert_allclose(st.logits[b], bf[b]["logits"][T + s], rtol=0, atol=1e-12)


def test_nan_poisoned_cache_slots_are_never_read(small):
    """Every cache slot a query reads was written (computed or generated):
    a run with exits produces finite logits and exactly layers i*+1..N of an
    exited token's slot are generated."""
    w, ids = small
    cfg = O.ExitConfig(delta=_quantile_delta(w, ids, "local", 2, 0.4), metric=O.LOCAL)
    res, cache = O.prefill(w, SMALL, ids, cfg)
    assert np.isfinite(res.logits).all()
    assert np.isfinite(cache.k).all() and np.isfinite(cache.v).all()


# --------------------------------------------------------------------------
# classification mode vs transformers' BERT
# --------------------------------------------------------------------------

ENC = ai.EncoderShape(n_layers=3, d_model=48, n_heads=3, head_dim=16, d_ff=96, vocab=101,
                      max_pos=32)


def test_classify_full_depth_matches_transformers_bert():
    w = O.as64(ai.encoder_weights(ENC, seed=21))
    ids = ai.token_ids(22, ENC.vocab, 3, 10)
    res = O.classify(w, ENC, ids, O.ExitConfig(delta=math.inf))
    m = hf_models.bert(ENC, w)
    with torch.no_grad():
        out = m(torch.from_numpy(ids.astype(np.int64))).last_hidden_state.numpy()
    np.testing.assert_allclose(res.h_final.reshape(out.shape), out, rtol=0, atol=1e-12)
    cls = out[:, 0] @ w["cls_w"].T + w["cls_b"]
    np.testing.assert_allclose(res.logits, cls, rtol=0, atol=1e-12)


def test_classify_exits_drop_tokens_from_later_keys():
    """With a forced exit schedule, each layer's output for the live tokens
    equals transformers' BERT layer run on the live tokens of each sequence
    alone (exited tokens no longer take part), and the [CLS] logits use the
    [CLS] state at its exit."""
    w = O.as64(ai.encoder_weights(ENC, seed=21))
    ids = ai.token_ids(23, ENC.vocab, 2, 8)
    force = np.random.default_rng(1).integers(0, ENC.n_layers + 1, size=ids.shape)
    res = O.classify(w, ENC, ids, O.ExitConfig(delta=math.inf), force_layer=force)
    m = hf_models.bert(ENC, w)
    B, T = ids.shape
    with torch.no_grad():
        h = m.embeddings(torch.from_numpy(ids.astype(np.int64)))
        ex = res.exit_layer.reshape(B, T)
        for i in range(1, ENC.n_layers + 1):
            for b in range(B):
                live = np.nonzero(ex[b] >= i)[0]
                if live.size == 0:
                    continue
                out = m.encoder.layer[i - 1](h[b:b + 1, live])
                out = out[0] if isinstance(out, tuple) else out
                h[b, live] = out[0]
    np.testing.assert_allclose(res.h_final.reshape(B, T, -1), h.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("force", [False, True])
def test_classify_stop_at_cls(force):
    """Stopping a sequence when its [CLS] row exits changes nothing the
    classifier sees: the logits are identical to the run that keeps the other
    tokens going, and each token's exit layer is the smaller of its own (in
    that run) and its [CLS] row's; with the policy, some tokens are stopped
    early and some exit on their own before their [CLS]."""
    w = O.as64(ai.encoder_weights(ENC, seed=24))
    ids = ai.token_ids(25, ENC.vocab, 4, 12)
    B, T = ids.shape
    fl = None
    if force:
        fl = np.random.default_rng(26).integers(0, ENC.n_layers + 1, size=ids.shape)
        fl[:, 0] = [1, 2, 3, 0]
        delta = math.inf
    else:
        full = O.classify(w, ENC, ids, O.ExitConfig(delta=math.inf), stop_at_cls=False)
        fin = np.sort(full.sims[:ENC.n_layers - 1][np.isfinite(full.sims[:ENC.n_layers - 1])])
        q = fin.size // 2
        delta = float(0.5 * (fin[q - 1] + fin[q]))      # between two similarities
    cfg = O.ExitConfig(delta=delta)
    go = O.classify(w, ENC, ids, cfg, force_layer=fl, stop_at_cls=False)
    st = O.classify(w, ENC, ids, cfg, force_layer=fl, stop_at_cls=True)
    # equal up to the summation order of the batched products (fewer rows)
    np.testing.assert_allclose(st.logits, go.logits, rtol=0, atol=1e-14)
    np.testing.assert_array_equal(st.cls_exit_layer, go.cls_exit_layer)
    el_go, el_st = go.exit_layer.reshape(B, T), st.exit_layer.reshape(B, T)
    np.testing.assert_array_equal(el_st, np.minimum(el_go, el_go[:, :1]))
    assert (el_st < el_go).any() and ((el_st < el_st[:, :1]).any() or force)


def test_cls_stop_rule():
    """cls_stop on a hand-made list: rows 0..3 are sequence 0, 4..7 sequence 1,
    8..11 sequence 2 (seq_len 4).  Sequence 0's [CLS] (row 0) exits now,
    sequence 1's [CLS] (row 4) has already left, sequence 2's stays."""
    active = np.array([0, 2, 3, 5, 7, 8, 9, 11])
    flags = np.array([1, 0, 0, 0, 0, 0, 1, 0], bool)
    out = O.cls_stop(flags, active, 4)
    np.testing.assert_array_equal(out, [1, 1, 1, 1, 1, 0, 1, 0])
    assert O.cls_stop(np.zeros(0, bool), np.zeros(0, np.int64), 4).size == 0


# --------------------------------------------------------------------------
# Section 6 accounting (values printed in the paper)
# --------------------------------------------------------------------------

def test_section6_accounting():
    g = json.load(open(os.path.join(GOLDEN, "section6_accounting.json")))
    x = g["gpt2_xl"]
    ex = np.full(1, g["exit_all_at_layer"])
    no_kv = acc.reduction(x["n_layers"], x["d_model"], x["d_ff"], x["vocab"], ex, "none")
    with_kv = acc.reduction(x["n_layers"], x["d_model"], x["d_ff"], x["vocab"], ex, "paper")
    # the printed figures are the percentages cut to one decimal (19.76 -> 19.7)
    for val, printed in ((no_kv, g["reduction_percent_without_kv_generation"]),
                         (with_kv, g["reduction_percent_with_kv_generation"])):
        assert printed <= 100 * val < printed + 0.1
    assert round(acc.exit_module_flops(x["d_model"], x["vocab"]) / 1e6) == \
        g["module_metric_mflops_per_token_per_layer"]
    be = acc.break_even_layer(x["n_layers"], g["regular_layer_mflops_per_token"],
                              g["module_metric_mflops_per_token_per_layer"])
    assert math.floor(be) == g["module_break_even_before_layer"]
    # no exit saves nothing; the algorithmic K+V charge is larger than the paper's
    assert acc.reduction(48, 1600, 6400, 50257, np.full(3, 48)) == 0.0
    assert acc.reduction(48, 1600, 6400, 50257, ex, "algorithmic") < with_kv


# --------------------------------------------------------------------------
# planted mistakes: each is caught by at least one pin above
# --------------------------------------------------------------------------

def _fails(fn, *args):
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


def test_planted_mistakes(small, monkeypatch):
    """Plant plausible mistakes in the oracle (on the CPU) and check that the
    pins catch each one."""
    real_rope, real_kv, real_attend = O.apply_rope, O.kv_generate, O.attend

    def rope_wrong_sign(x, pos, theta):
        hd = x.shape[-1]
        c, s = O.rope_cos_sin(pos, hd, theta)
        x1, x2 = x[..., : hd // 2], x[..., hd // 2:]
        return np.concatenate([x1 * c[:, None] + x2 * s[:, None], x2 * c[:, None] - x1 * s[:, None]], -1)

    def kv_one_layer_early(weights, shape, s_map, exit_layer, pos):
        return real_kv(weights, shape, s_map, np.asarray(exit_layer) - 1, pos)

    def attend_drops_own_key(q, k, v, base, pos, *a, **kw):
        return real_attend(q, k, v, base, np.maximum(np.asarray(pos) - 1, 0), *a, **kw)

    def inertia_before_test(inertia, h):
        return np.asarray(inertia, F64) * 0.0 + np.asarray(h, F64) / np.linalg.norm(h, axis=1, keepdims=True)

    F64 = np.float64
    planted = [
        ("apply_rope", rope_wrong_sign, test_full_depth_matches_transformers_llama),
        ("kv_generate", kv_one_layer_early,
         lambda s: test_batched_prefill_equals_token_at_a_time(s, "local", 2, 0.5, False)),
        ("attend", attend_drops_own_key, test_full_depth_matches_transformers_llama),
        ("inertia_update", inertia_before_test, test_inertia_is_sum_of_unit_states),
    ]
    for name, bad, pin in planted:
        with monkeypatch.context() as mp:
            mp.setattr(O, name, bad)
            assert _fails(pin, small), f"planted mistake in {name} was not caught"
    assert O.apply_rope is real_rope
