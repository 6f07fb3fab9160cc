"""Pins of the oracle's GPT-2-family decoder (LayerNorm with bias, learned
positions, tanh GELU, biases, tied head) on the CPU: transformers' GPT-2 in
fp64 is an independent statement of the base model's layers; the early-exit
machinery around the layers is the same code as for the llama family."""
import math

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import adept_oracle as O
from tests import hf_models

SHAPE = ai.DecoderShape(n_layers=4, d_model=96, n_heads=3, head_dim=32, d_ff=384, vocab=160,
                        family="gpt2", max_pos=64)


@pytest.fixture(scope="module")
def gp():
    w = O.as64(ai.gpt2_weights(SHAPE, seed=3, dtype="f32", std=0.05))
    ids = ai.token_ids(4, SHAPE.vocab, 2, 24)
    return w, ids


def test_gelu_tanh_matches_torch():
    x = np.linspace(-6, 6, 1001)
    want = torch.nn.functional.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    np.testing.assert_allclose(O.gelu_tanh(x), want, rtol=0, atol=1e-15)


def test_full_depth_matches_transformers_gpt2(gp):
    """delta = +inf: logits and the K/V cache equal transformers'
    GPT2LMHeadModel in fp64."""
    w, ids = gp
    res, cache = O.prefill(w, SHAPE, ids, O.ExitConfig(delta=math.inf))
    m = hf_models.gpt2(SHAPE, w)
    with torch.no_grad():
        out = m(torch.from_numpy(ids.astype(np.int64)), use_cache=True)
    B, T = ids.shape
    np.testing.assert_allclose(res.logits.reshape(B, T, -1), out.logits.numpy(), rtol=0,
                               atol=1e-11)
    for i in range(SHAPE.n_layers):
        hk = out.past_key_values.layers[i].keys.numpy()      # [B, H, T, hd]
        hv = out.past_key_values.layers[i].values.numpy()
        ok = cache.k[i].reshape(B, T, SHAPE.n_heads, SHAPE.head_dim).transpose(0, 2, 1, 3)
        ov = cache.v[i].reshape(B, T, SHAPE.n_heads, SHAPE.head_dim).transpose(0, 2, 1, 3)
        np.testing.assert_allclose(ok, hk, rtol=0, atol=1e-12)
        np.testing.assert_allclose(ov, hv, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_exit_everything_at_k_gpt2(gp, k):
    """Every token exits at layer k (delta = -1, local metric, minimum exit
    layer k): the logits are the k-layer truncated model's (its final
    LayerNorm and tied head on h_k), and the generated K/V of every layer
    r > k are transformers' layer-r LayerNorm and c_attn key / value path
    applied to h_k (Eq. 9 with the identity mapper)."""
    w, ids = gp
    res, cache = O.prefill(w, SHAPE, ids, O.ExitConfig(delta=-1.0, min_exit_layer=k,
                                                       metric=O.LOCAL))
    assert (res.exit_layer == k).all()
    B, T = ids.shape
    tid = torch.from_numpy(ids.astype(np.int64))
    trunc = hf_models.gpt2(SHAPE, w, n_layers=k)
    with torch.no_grad():
        out = trunc(tid)
    np.testing.assert_allclose(res.logits.reshape(B, T, -1), out.logits.numpy(), rtol=0,
                               atol=1e-11)
    full = hf_models.gpt2(SHAPE, w)
    H, hd, D = SHAPE.n_heads, SHAPE.head_dim, SHAPE.d_model
    with torch.no_grad():
        hk = full(tid, output_hidden_states=True).hidden_states[k]   # input of layer k+1
        for r in range(k + 1, SHAPE.n_layers + 1):
            L = full.transformer.h[r - 1]
            qkv = L.attn.c_attn(L.ln_1(hk))
            kk = qkv[..., D:2 * D].reshape(B, T, H, hd).numpy()
            vv = qkv[..., 2 * D:].reshape(B, T, H, hd).numpy()
            np.testing.assert_allclose(cache.k[r - 1].reshape(B, T, H, hd), kk, rtol=0, atol=1e-12)
            np.testing.assert_allclose(cache.v[r - 1].reshape(B, T, H, hd), vv, rtol=0, atol=1e-12)


@pytest.mark.parametrize("metric", ["global", "local"])
def test_batched_prefill_equals_token_at_a_time_gpt2(gp, metric):
    """The batched prefill with compaction and decoupled KV generation equals
    feeding the prompt one token at a time (each a one-row pass over the
    cache the earlier tokens filled), at a threshold that fires: same exit
    layers, logits and caches (causality makes the two equal)."""
    w, ids = gp
    full, _ = O.prefill(w, SHAPE, ids, O.ExitConfig(delta=math.inf, metric=metric))
    s = np.sort(full.sims[:SHAPE.n_layers - 1][np.isfinite(full.sims[:SHAPE.n_layers - 1])])
    j = int(0.9 * len(s))
    delta = float(0.5 * (s[j] + s[j + 1]))
    cfg = O.ExitConfig(delta=delta, metric=metric)
    res, cache = O.prefill(w, SHAPE, ids, cfg)
    assert 0 < np.sum(res.exit_layer < SHAPE.n_layers) < res.exit_layer.size
    B, T = ids.shape
    seq_cache = O.KVCache.empty(SHAPE, B, T)
    logits, el = [], []
    for t in range(T):
        st = O.decode_step(w, SHAPE, seq_cache, ids[:, t], np.full(B, t), cfg)
        logits.append(st.logits)
        el.append(st.exit_layer)
    np.testing.assert_array_equal(np.stack(el, axis=1).reshape(-1), res.exit_layer)
    np.testing.assert_allclose(np.stack(logits, axis=1).reshape(B * T, -1), res.logits, rtol=0,
                               atol=1e-12)
    np.testing.assert_allclose(seq_cache.k, cache.k, rtol=0, atol=1e-12)
    np.testing.assert_allclose(seq_cache.v, cache.v, rtol=0, atol=1e-12)


def test_gpt2_xl_accounting_shape():
    """The GPT2-XL shape of Section 6 (48 layers, width 1600) is the shape the
    paper's compute-reduction figures use."""
    assert (ai.GPT2_XL.n_layers, ai.GPT2_XL.d_model, ai.GPT2_XL.d_q) == (48, 1600, 1600)
