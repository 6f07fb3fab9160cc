"""GPU parity of the LayerNorm decoder family (GPT-2 style; the GPT2-XL shape
of Section 5) against the oracle.

Every layer is checked teacher-forced on the GPU's own inputs (tests/
layer_check.py): the LayerNorm, the biased Q/K/V projections (their gain and
shift folded into the weights and bias), the attention over the mixed cache,
the biased output projection, the tanh-GELU MLP, the exit test and the list
update; after the pass the K/V generated for exited tokens from their exit
state through the skipped layers' LayerNorm and biased K/V projections
(Eq. 9) and the logits of the final LayerNorm and the tied head.

The small shape has ragged column tiles everywhere (width 320 = 5 heads of
64: Q/K/V 960 columns, 3.75 tiles of 256; output and second MLP projection
320 columns; first MLP projection 1280); the GPT2-XL-width cases run the
real layer shapes (width 1600, 25 heads, MLP 6400) with fewer layers.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import adept_oracle as O
from paper_2601_03700_amd import binding as B
from paper_2601_03700_amd.calibrate import SimRecorder, running_max
from paper_2601_03700_amd.model import DecoderModel
from tests import layer_check as LC

pytestmark = pytest.mark.gpu

SMALL = ai.DecoderShape(n_layers=5, d_model=320, n_heads=5, head_dim=64, d_ff=1280, vocab=576,
                        family="gpt2", max_pos=512)
XL_3L = ai.DecoderShape(n_layers=3, d_model=1600, n_heads=25, head_dim=64, d_ff=6400, vocab=512,
                        family="gpt2", max_pos=1024)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def w_small():
    w = ai.gpt2_weights(SMALL, seed=41, dtype="bf16")
    return w, O.as64(w)


@pytest.fixture(scope="module")
def w_xl():
    w = ai.gpt2_weights(XL_3L, seed=42, dtype="bf16")
    return w, O.as64(w)


def _half_forced(seed, shape_ids, n_layers):
    rng = np.random.default_rng(seed)
    f = rng.integers(1, n_layers + 1, size=shape_ids)
    return np.where(rng.random(shape_ids) < 0.5, 0, f).astype(np.int32)


def _firing_delta(model, ids, metric, frac):
    """A threshold that makes the policy exit about `frac` of the
    (token, tested layer) pairs: from the similarities of a pass that never
    exits, half-way between two neighbouring running maxima (so that no
    similarity sits on the threshold)."""
    N = model.shape.n_layers
    rec = SimRecorder(N, ids.size, model.device)
    model.prefill(ids, B.exit_cfg(math.inf, N, metric), logits=None, on_layer=rec)
    m = np.sort(running_max(rec.sims.cpu().numpy(), N).ravel())[::-1]
    m = m[np.isfinite(m)]
    k = max(1, int(frac * m.size))
    lo = m[k:][m[k:] < m[k - 1] - 1e-9]
    return float((m[k - 1] + lo[0]) / 2) if lo.size else float(m[k - 1] - 1e-6)


def _tf_prefill(model, w, shape, ids, delta, metric, force, rep, s_max=None, logits="all"):
    chk = LC.DecoderLayerCheck(w, shape, None, O.ExitConfig(delta=delta, metric=metric), "bf16",
                               force_layer=force, report=rep)
    cache = model.new_cache(ids.shape[0], ids.shape[1] if s_max is None else s_max)
    chk.cache = cache
    res, cache = model.prefill(ids, B.exit_cfg(delta, shape.n_layers, metric), s_max=s_max,
                               force_layer=force, logits=logits, cache=cache, on_layer=chk)
    chk.finish(res.state, res.logits, res.rows)
    return res, cache, chk


def _tf_decode(model, w, shape, cache, ids, pos, delta, metric, force, rep):
    chk = LC.DecoderLayerCheck(w, shape, cache, O.ExitConfig(delta=delta, metric=metric), "bf16",
                               force_layer=force, report=rep)
    dev = model.device
    res = model.decode_step(cache, torch.from_numpy(np.asarray(ids)).to(dev, torch.int32),
                            torch.from_numpy(np.asarray(pos)).to(dev, torch.int32),
                            B.exit_cfg(delta, shape.n_layers, metric),
                            force_layer=torch.from_numpy(np.asarray(force)).to(dev, torch.int32),
                            on_layer=chk)
    chk.finish(res.state, res.logits, res.rows)
    return res, chk


def test_gpt2_embed_positions(w_small):
    """h_0 = wte[id] + wpe[pos], summed in f32 and rounded once to bf16,
    against the oracle's embedding (including ids and positions at the table
    ends)."""
    w, w64 = w_small
    s = SMALL
    n = 300
    rng = np.random.default_rng(5)
    ids = rng.integers(0, s.vocab, n).astype(np.int32)
    pos = rng.integers(0, s.max_pos, n).astype(np.int32)
    ids[:2], pos[:2] = [0, s.vocab - 1], [s.max_pos - 1, 0]
    dev = torch.device("cuda")
    wte = torch.from_numpy(np.asarray(w["embed"], np.float32)).to(dev, torch.bfloat16)
    wpe = torch.from_numpy(np.asarray(w["pos_embed"], np.float32)).to(dev, torch.bfloat16)
    h0 = torch.empty((n, s.d_model), dtype=torch.bfloat16, device=dev)
    B.embed_positions(n, s.d_model, s.vocab, s.max_pos, torch.from_numpy(ids).to(dev),
                      torch.from_numpy(pos).to(dev), wte, wpe, h0)
    torch.cuda.synchronize()
    rep = LC.Report(say)
    rep.check("h_0", LC.host(h0), O.embed_rows(w64, s, ids, pos), "bf16")
    rep.summary()


def test_gpt2_fold_bias():
    """bias += W beta per matrix of a stack (the LayerNorm shift folded into
    the projection's bias), against the fp64 product, within one bf16
    rounding of the result."""
    rng = np.random.default_rng(6)
    L, rows, cols = 3, 200, 320
    w = ai.to_bf16_values(rng.normal(0, 0.02, (L, rows, cols)))
    beta = ai.to_bf16_values(rng.normal(0, 0.5, (L, cols)))
    b = ai.to_bf16_values(rng.normal(0, 0.02, (L, rows)))
    dev = torch.device("cuda")
    tw, tbeta, tb = (torch.from_numpy(np.asarray(x, np.float32)).to(dev, torch.bfloat16)
                     for x in (w, beta, b))
    B.fold_bias(tw, tbeta, tb)
    torch.cuda.synchronize()
    want = b + np.einsum("lrc,lc->lr", w.astype(np.float64), beta.astype(np.float64))
    got = LC.host(tb)
    assert np.all(np.abs(got - want) <= np.maximum(np.abs(want) * 2.0 ** -8, 1e-6))


@pytest.mark.parametrize("metric", ["global", "local"])
def test_gpt2_small_prefill_teacher_forced(w_small, metric):
    """Prefill of 3 x 200 rows at the ragged small shape, half of the rows on a
    seeded exit schedule and half on the policy at a threshold that exits
    about a fifth of the token-layers: every layer checked on the GPU's own
    inputs, then the generated K/V of the exited rows and all logits."""
    say(f"gpt2 small prefill teacher-forced metric={metric}")
    w, w64 = w_small
    ids = ai.token_ids(43, SMALL.vocab, 3, 200)
    model = DecoderModel(SMALL, w, dtype="bf16")
    delta = _firing_delta(model, ids, metric, 0.2)
    force = _half_forced(44, ids.shape, SMALL.n_layers)
    rep = LC.Report(say)
    res, cache, chk = _tf_prefill(model, w64, SMALL, ids, delta, metric, force, rep)
    rep.summary()
    el = chk.exit_layer
    policy_exits = int(np.sum((force.reshape(-1) == 0) & (el < SMALL.n_layers)))
    say(f"  delta {delta:.6f}: exits {int(np.sum(el < SMALL.n_layers))} of {el.size} "
        f"(policy {policy_exits})")
    assert policy_exits > 0 and np.sum(el == SMALL.n_layers) > 0


@pytest.mark.parametrize("kv_fused", [True, False])
def test_gpt2_small_decode_teacher_forced(w_small, kv_fused):
    """Decode at the small shape: a prompt of 24 sequences x 9 rows, then one
    step per sequence (skinny GEMMs with biases and the tanh-GELU epilogue,
    key-chunked attention, the deferred LayerNorm KV generation), both
    checked layer by layer; then a second step over the generated entries."""
    say(f"gpt2 small decode teacher-forced kv_fused={kv_fused}")
    w, w64 = w_small
    N = SMALL.n_layers
    Bn, T = 24, 9
    ids = ai.token_ids(45, SMALL.vocab, Bn, T)
    rng = np.random.default_rng(46)
    force_p = rng.integers(0, N + 1, size=ids.shape).astype(np.int32)
    model = DecoderModel(SMALL, w, dtype="bf16", kv_fused=kv_fused)
    rep = LC.Report(say)
    _, cache, _ = _tf_prefill(model, w64, SMALL, ids, math.inf, "global", force_p, rep,
                              s_max=T + 2, logits="last")
    for k in range(2):
        step = ai.token_ids(47 + k, SMALL.vocab, 1, Bn)[0]
        force_s = rng.integers(1, N + 1, size=Bn).astype(np.int32)
        _, chk = _tf_decode(model, w64, SMALL, cache, step, np.full(Bn, T + k), math.inf,
                            "global", force_s, rep)
        assert np.sum(chk.exit_layer < N) > 0
    rep.summary()


@pytest.mark.parametrize("metric", ["global", "local"])
def test_gpt2_small_free_running_decisions(w_small, metric):
    """The policy end to end (no teacher forcing): a threshold half-way between
    two of the oracle's similarities of a pass without exits; every token whose
    oracle margin |sim - delta| exceeds 5e-3 at all its tested layers exits at
    the same layer on the GPU."""
    say(f"gpt2 small free running metric={metric}")
    w, w64 = w_small
    ids = ai.token_ids(54, SMALL.vocab, 2, 128)
    N = SMALL.n_layers
    full, _ = O.prefill(w64, SMALL, ids, O.ExitConfig(delta=math.inf, metric=metric))
    sims = np.sort(full.sims[:N - 1][np.isfinite(full.sims[:N - 1])])
    q = int((0.6 if metric == "global" else 0.9) * sims.size)   # both: some tokens never exit
    delta = float(0.5 * (sims[q] + sims[q + 1]))
    model = DecoderModel(SMALL, w, dtype="bf16")
    res_g, _ = model.prefill(ids, B.exit_cfg(delta, N, metric), logits="all")
    torch.cuda.synchronize()
    res_o, _ = O.prefill(w64, SMALL, ids, O.ExitConfig(delta=delta, metric=metric))
    el_g, el_o = res_g.exit_layer.cpu().numpy(), res_o.exit_layer
    m = np.abs(res_o.sims - delta)
    safe = np.nanmin(np.where(np.isfinite(m), m, np.inf), axis=0) > 5e-3
    say(f"  delta {delta:.6f}: {int(safe.sum())} of {safe.size} tokens decided with margin, "
        f"{int(np.sum(el_o < N))} exits")
    assert safe.sum() > 0.3 * safe.size and 0 < np.sum(el_o < N) < el_o.size
    np.testing.assert_array_equal(el_g[safe], el_o[safe])


def test_gpt2_xl_width_prefill_teacher_forced(w_xl):
    """Prefill at the GPT2-XL layer shapes (width 1600, 25 heads of 64, MLP
    6400; three layers): 2 x 520 rows (five 256-row tiles, the last ragged;
    Q/K/V 4800 columns = 18.75 tiles), half forced, half on the policy."""
    say("gpt2-xl width prefill teacher-forced")
    w, w64 = w_xl
    ids = ai.token_ids(48, XL_3L.vocab, 2, 520)
    model = DecoderModel(XL_3L, w, dtype="bf16")
    delta = _firing_delta(model, ids, "global", 0.2)
    force = _half_forced(49, ids.shape, XL_3L.n_layers)
    rep = LC.Report(say)
    _, _, chk = _tf_prefill(model, w64, XL_3L, ids, delta, "global", force, rep)
    rep.summary()
    el = chk.exit_layer
    say(f"  delta {delta:.6f}: exits {int(np.sum(el < XL_3L.n_layers))} of {el.size}")
    assert 0 < np.sum(el < XL_3L.n_layers) < el.size


def test_gpt2_xl_width_decode_teacher_forced(w_xl):
    """Decode at the GPT2-XL layer shapes, 48 sequences: the skinny GEMMs at
    K = 1600 and 6400 with ragged stream-K ranges, the deferred generation."""
    say("gpt2-xl width decode teacher-forced")
    w, w64 = w_xl
    N = XL_3L.n_layers
    Bn, T = 48, 3
    ids = ai.token_ids(50, XL_3L.vocab, Bn, T)
    rng = np.random.default_rng(51)
    force_p = rng.integers(0, N + 1, size=ids.shape).astype(np.int32)
    force_s = rng.integers(1, N + 1, size=Bn).astype(np.int32)
    model = DecoderModel(XL_3L, w, dtype="bf16")
    rep = LC.Report(say)
    _, cache, _ = _tf_prefill(model, w64, XL_3L, ids, math.inf, "global", force_p, rep,
                              s_max=T + 1, logits="last")
    step = ai.token_ids(52, XL_3L.vocab, 1, Bn)[0]
    _, chk = _tf_decode(model, w64, XL_3L, cache, step, np.full(Bn, T), math.inf, "global",
                        force_s, rep)
    rep.summary()
    assert np.sum(chk.exit_layer < N) > 0


def test_gpt2_kv_generate_layernorm_direct(w_small):
    """adept_kv_generate_layernorm called alone on a ragged list (rows in
    descending order, exit layers 1..N-1 and one that never exited), against
    the oracle's Eq. 9 for the LayerNorm family; untouched slots stay as they
    were, and an empty list writes nothing."""
    w, w64 = w_small
    s = SMALL
    N, D, H, hd = s.n_layers, s.d_model, s.n_heads, s.head_dim
    model = DecoderModel(s, w, dtype="bf16")
    dev = model.device
    n_tok = 70
    rng = np.random.default_rng(53)
    s_map = ai.to_bf16_values(rng.normal(0, 1.0, (n_tok, D)))
    exit_layer = rng.integers(1, N + 1, n_tok).astype(np.int32)
    pos = np.arange(n_tok, dtype=np.int64)
    rows = np.sort(rng.choice(n_tok, 45, replace=False))[::-1].astype(np.int32)
    slot = np.arange(n_tok, dtype=np.int32)
    cache = model.new_cache(1, n_tok, fill=7.0)
    t = lambda x, dt=torch.int32: torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)
    s_t = torch.from_numpy(s_map.astype(np.float32)).to(dev, torch.bfloat16)
    ws = torch.empty(B.kv_generate_layernorm_workspace_bytes(N, n_tok, D), dtype=torch.uint8,
                     device=dev)
    esz = 2
    dq = H * hd
    w_kv = model.w_qkv.data_ptr() + dq * D * esz
    b_kv = model.b_qkv.data_ptr() + dq * esz
    n0 = t(np.array([0], np.int32))
    B.kv_generate_layernorm(N, D, H, hd, s.ln_eps, s_t, t(rows), n0, n_tok, t(exit_layer),
                            t(slot), w_kv, 3 * dq * D, b_kv, 3 * dq, cache.k, cache.v,
                            cache.n_slots, ws)
    torch.cuda.synchronize()
    assert bool((cache.k.float() == 7.0).all()) and bool((cache.v.float() == 7.0).all())
    B.kv_generate_layernorm(N, D, H, hd, s.ln_eps, s_t, t(rows), t(np.array([rows.size], np.int32)),
                            n_tok, t(exit_layer), t(slot), w_kv, 3 * dq * D, b_kv, 3 * dq,
                            cache.k, cache.v, cache.n_slots, ws)
    torch.cuda.synchronize()
    gen = O.kv_generate(w64, s, s_map[rows].astype(np.float64), exit_layer[rows], pos[rows])
    kc, vc = LC.host(cache.k), LC.host(cache.v)
    rep = LC.Report(say)
    touched = np.zeros((N, n_tok), bool)
    for r, (idx, k, v) in gen.items():
        sl = slot[rows[idx]]
        rep.check(f"K (generated)@{r}", kc[r - 1][sl], k, "bf16")
        rep.check(f"V (generated)@{r}", vc[r - 1][sl], v, "bf16")
        touched[r - 1, sl] = True
    rep.summary()
    assert np.all(kc[~touched] == 7.0) and np.all(vc[~touched] == 7.0)
