"""End-to-end parity of the early-exit forward (prefill + generation) on the
GPU against the oracle, through adept_layer_step and the support calls.

fp32 (the tiny 4-layer configuration): free-running; exit layers must match
exactly and logits / caches within 1e-5 relative (max-norm).  bf16: teacher-
forced per layer (tests/layer_check.py): each layer's GPU input goes to the
oracle's layer and its outputs are compared per element within max(2e-2,
one bf16 ulp); exit flags, lists and exit layers bit-exactly on identical
inputs; free-running bf16 decisions end to end are compared where the
oracle's margin |sim - delta| exceeds the bf16 error.
"""
import math
import sys

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import adept_oracle as O
from paper_2601_03700_amd import binding as B
from paper_2601_03700_amd.model import DecoderModel
from tests import layer_check as LC

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))


def cache_host(cache, B_, T):
    k = cache.k.float().cpu().numpy().astype(np.float64)
    v = cache.v.float().cpu().numpy().astype(np.float64)
    return k, v


def oracle_deltas(w, shape, ids, metric):
    """Thresholds that fire for part of the tokens: quantiles of the oracle's
    similarities at layers 1..N-1 of a run that never exits."""
    res, _ = O.prefill(w, shape, ids, O.ExitConfig(delta=math.inf, metric=metric))
    s = res.sims[: shape.n_layers - 1]
    s = np.sort(s[np.isfinite(s)])
    # midpoints between neighbouring similarities, so no token sits on delta
    return [float(0.5 * (s[int(q * len(s))] + s[int(q * len(s)) + 1])) for q in (0.5, 0.8)]


TINY = ai.TINY


@pytest.fixture(scope="module")
def tiny_f32():
    w = ai.decoder_weights(TINY, seed=1, dtype="f32")
    ids = ai.token_ids(2, TINY.vocab, 1, 128)
    model = DecoderModel(TINY, w, dtype="f32", rope_max_pos=256)
    return O.as64(w), ids, model


@pytest.mark.parametrize("metric", ["local", "global", "both"])
def test_tiny_f32_prefill_and_decode(tiny_f32, metric):
    """The tiny configuration (4 layers, width 256, 128-token prompt, 32
    greedy steps, local metric at delta 0.95) and thresholds that fire."""
    w, ids, model = tiny_f32
    deltas = [0.95] + oracle_deltas(w, TINY, ids, metric)
    for delta in deltas:
        say(f"tiny f32 metric={metric} delta={delta:.6f}")
        cfg_o = O.ExitConfig(delta=delta, metric=metric)
        cfg_g = B.exit_cfg(delta, TINY.n_layers, metric)
        n_steps = 32
        res_o, steps_o, gen_o, cache_o = O.generate(w, TINY, ids, n_steps, cfg_o)
        res_g, cache_g = model.prefill(ids, cfg_g, s_max=128 + n_steps, logits="all")
        torch.cuda.synchronize()
        el_g = res_g.exit_layer.cpu().numpy()
        # margin check: no oracle similarity within 1e-6 of delta (f32 state)
        tested = res_o.sims[: TINY.n_layers - 1]
        margin = np.nanmin(np.abs(tested - delta)) if np.isfinite(tested).any() else np.inf
        assert margin > 1e-6, f"delta {delta} too close to a similarity ({margin})"
        np.testing.assert_array_equal(el_g, res_o.exit_layer)
        assert rel_err(res_g.logits.cpu().numpy(), res_o.logits) <= 1e-5
        # greedy decode on the GPU, compared step by step
        nxt = model.greedy(res_g.logits[-1:].contiguous())
        for s in range(n_steps):
            assert int(nxt[0]) == int(gen_o[0, s]), f"step {s}"
            pos = torch.full((1,), 128 + s, dtype=torch.int32, device="cuda")
            st = model.decode_step(cache_g, nxt, pos, cfg_g)
            torch.cuda.synchronize()
            assert int(st.exit_layer[0]) == int(steps_o[s].exit_layer[0]), f"step {s}"
            assert rel_err(st.logits.cpu().numpy(), steps_o[s].logits) <= 1e-5
            nxt = model.greedy(st.logits)
        kg, vg = cache_host(cache_g, 1, 128 + n_steps)
        assert rel_err(kg, cache_o.k) <= 1e-5 and rel_err(vg, cache_o.v) <= 1e-5


@pytest.mark.parametrize("metric", ["global", "local"])
def test_tiny_f32_all_at_once_prefill(metric):
    """All-at-once variant (Appendix H.2) on the GPU: every prompt's tokens
    take the decision of its last token; exit layers exact, logits and the
    K/V cache within the f32 bound."""
    w32 = ai.decoder_weights(TINY, seed=4, dtype="f32")
    w = O.as64(w32)
    ids = ai.token_ids(6, TINY.vocab, 4, 40)
    B_, T = ids.shape
    model = DecoderModel(TINY, w32, dtype="f32", rope_max_pos=64)
    full, _ = O.prefill(w, TINY, ids, O.ExitConfig(delta=math.inf, metric=metric))
    s_last = full.sims[: TINY.n_layers - 1, np.arange(B_) * T + T - 1]
    s = np.sort(s_last[np.isfinite(s_last)])
    for q in (0.4, 0.7):
        j = int(q * (len(s) - 1))
        delta = float(0.5 * (s[j] + s[j + 1]))
        say(f"all-at-once metric={metric} delta={delta:.6f}")
        cfg_o = O.ExitConfig(delta=delta, metric=metric, prompt_level=True)
        res_o, cache_o = O.prefill(w, TINY, ids, cfg_o, s_max=T)
        res_g, cache_g = model.prefill(ids, B.exit_cfg(delta, TINY.n_layers, metric,
                                                       prompt_level=True), s_max=T, logits="all")
        torch.cuda.synchronize()
        tested = res_o.sims[: TINY.n_layers - 1]
        assert np.nanmin(np.abs(tested - delta)) > 1e-6
        el = res_g.exit_layer.cpu().numpy()
        np.testing.assert_array_equal(el, res_o.exit_layer)
        for b in range(B_):      # one exit layer per prompt
            assert len(set(el[b * T:(b + 1) * T].tolist())) == 1
        assert rel_err(res_g.logits.cpu().numpy(), res_o.logits) <= 1e-5
        kg, vg = cache_host(cache_g, B_, T)
        assert rel_err(kg, cache_o.k) <= 1e-5 and rel_err(vg, cache_o.v) <= 1e-5


SMALL_BF16 = ai.DecoderShape(n_layers=6, d_model=512, n_heads=4, head_dim=128, d_ff=1024,
                             vocab=512)


def _tf_prefill(model, w, shape, ids, cfg_o, cfg_g, force=None, s_max=None, logits="all",
                n_sample=256, rep=None):
    """Prefill on the GPU with the teacher-forced per-layer check, then the
    generated K/V and the logits of the GPU's final states."""
    chk = LC.DecoderLayerCheck(w, shape, None, cfg_o, model.dtype, force_layer=force,
                               n_sample=n_sample, report=rep)
    cache = model.new_cache(ids.shape[0], ids.shape[1] if s_max is None else s_max)
    chk.cache = cache
    res, cache = model.prefill(ids, cfg_g, s_max=s_max, force_layer=force, logits=logits,
                               cache=cache, on_layer=chk)
    chk.finish(res.state, res.logits, res.rows)
    return res, cache, chk


def _tf_decode(model, w, shape, cache, ids, pos, cfg_o, cfg_g, force=None, rep=None):
    chk = LC.DecoderLayerCheck(w, shape, cache, cfg_o, model.dtype, force_layer=force,
                               report=rep)
    dev = model.device
    res = model.decode_step(cache, torch.from_numpy(np.asarray(ids)).to(dev, torch.int32),
                            torch.from_numpy(np.asarray(pos)).to(dev, torch.int32), cfg_g,
                            force_layer=None if force is None else
                            torch.from_numpy(np.asarray(force)).to(dev, torch.int32),
                            on_layer=chk)
    chk.finish(res.state, res.logits, res.rows)
    return res, chk


def _half_forced(seed, shape_ids, n_layers):
    """Teacher-forced exit layers for about half of the rows (1..N, N = never),
    the policy's own decision (0) for the others."""
    rng = np.random.default_rng(seed)
    f = rng.integers(1, n_layers + 1, size=shape_ids)
    return np.where(rng.random(shape_ids) < 0.5, 0, f).astype(np.int32)


@pytest.mark.parametrize("metric", ["global", "local", "both"])
def test_small_bf16_prefill_teacher_forced(metric):
    """bf16 prefill (6 layers, width 512, 3 x 200 rows), half of the rows on a
    seeded exit schedule and half on the policy at a threshold that fires:
    every layer checked on the GPU's own inputs at the per-element bound."""
    say(f"small bf16 prefill teacher-forced metric={metric}")
    shape = SMALL_BF16
    w32 = ai.decoder_weights(shape, seed=9, dtype="bf16", std=0.03)
    w = O.as64(w32)
    ids = ai.token_ids(10, shape.vocab, 3, 200)
    force = _half_forced(5, ids.shape, shape.n_layers)
    delta = oracle_deltas(w, shape, ids, metric)[0]
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=512)
    rep = LC.Report(say)
    res, cache, chk = _tf_prefill(model, w, shape, ids, O.ExitConfig(delta=delta, metric=metric),
                                  B.exit_cfg(delta, shape.n_layers, metric), force=force, rep=rep)
    rep.summary()
    el = chk.exit_layer
    policy_exits = int(np.sum((force.reshape(-1) == 0) & (el < shape.n_layers)))
    say(f"  exits {int(np.sum(el < shape.n_layers))} (policy {policy_exits})")
    assert policy_exits > 0 and np.sum(el < shape.n_layers) < el.size


@pytest.mark.parametrize("kv_fused", [True, False])
def test_small_bf16_decode_teacher_forced(kv_fused):
    """bf16 generation: a prompt with a seeded schedule, then six decode
    passes (one row per sequence: key-chunked attention, skinny GEMMs, the
    K/V of exited rows from the later layers' QKV GEMMs or deferred to one
    grouped generation after the last layer), each pass checked layer by
    layer on the GPU's own inputs, generated K/V included."""
    say(f"small bf16 decode teacher-forced kv_fused={kv_fused}")
    shape = SMALL_BF16
    N = shape.n_layers
    w32 = ai.decoder_weights(shape, seed=9, dtype="bf16", std=0.03)
    w = O.as64(w32)
    Bn, T, S = 3, 40, 6
    ids = ai.token_ids(12, shape.vocab, Bn, T)
    step_ids = ai.token_ids(13, shape.vocab, S, Bn)
    rng = np.random.default_rng(6)
    force_p = rng.integers(0, N + 1, size=ids.shape).astype(np.int32)
    force_s = rng.integers(1, N + 1, size=(S, Bn)).astype(np.int32)   # every step token exits
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=512, kv_fused=kv_fused)
    cfg_g = B.exit_cfg(math.inf, N, "global")
    cfg_o = O.ExitConfig(delta=math.inf)
    rep = LC.Report(say)
    _, cache, _ = _tf_prefill(model, w, shape, ids, cfg_o, cfg_g, force=force_p, s_max=T + S,
                              logits="last", rep=rep)
    for s in range(S):
        _tf_decode(model, w, shape, cache, step_ids[s], np.full(Bn, T + s), cfg_o, cfg_g,
                   force=force_s[s], rep=rep)
    rep.summary()


def test_small_bf16_free_running_decisions():
    """bf16, policy-driven (global metric) end to end: every exit decision the
    oracle takes with a margin above the bf16 error of the similarity matches."""
    say("small bf16 free running")
    shape = SMALL_BF16
    w32 = ai.decoder_weights(shape, seed=9, dtype="bf16", std=0.03)
    w = O.as64(w32)
    ids = ai.token_ids(11, shape.vocab, 2, 128)
    delta = oracle_deltas(w, shape, ids, "global")[0]
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=512)
    res_g, _ = model.prefill(ids, B.exit_cfg(delta, shape.n_layers, "global"), logits="all")
    torch.cuda.synchronize()
    res_o, _ = O.prefill(w, shape, ids, O.ExitConfig(delta=delta, metric="global"))
    el_g, el_o = res_g.exit_layer.cpu().numpy(), res_o.exit_layer
    # a token is decided safely if at every layer it was tested its margin is > 5e-3
    m = np.abs(res_o.sims - delta)
    safe = np.nanmin(np.where(np.isfinite(m), m, np.inf), axis=0) > 5e-3
    assert safe.sum() > 0.5 * safe.size
    np.testing.assert_array_equal(el_g[safe], el_o[safe])
    assert 0 < np.sum(el_o < shape.n_layers) < el_o.size


SHAPE_7B_4L = ai.DecoderShape(n_layers=4, d_model=4096, n_heads=32, head_dim=128, d_ff=11008,
                              vocab=512)


@pytest.fixture(scope="module")
def w7b():
    """Four layers of the 7B-class decoder (width 4096, 32 x 128 heads, FFN
    11008; a 512-entry vocabulary) as bf16 values, and their float64 copy."""
    w32 = ai.decoder_weights(SHAPE_7B_4L, seed=21, dtype="bf16")
    return w32, O.as64(w32)


def test_7b_prefill_teacher_forced(w7b):
    """Prefill at the 7B layer shapes: 4 sequences x 600 rows (2400 rows: ten
    256-row GEMM tiles, the last ragged, at K = 4096 and K = 11008; 32 heads,
    so the query-tile attention takes its XCD-major one-dimensional grid, with
    a ragged last query tile per sequence).  Half of the rows follow a seeded
    schedule, half the policy; every layer is checked on the GPU's own
    inputs (>= 256 sampled rows for q, attention and h; all rows for K/V,
    exit flags, lists and exit layers), then the generated K/V of up to 256
    exited rows at all their skipped layers, and the logits."""
    shape = SHAPE_7B_4L
    say("7B-shape prefill teacher-forced (4 x 600 rows)")
    w32, w = w7b
    ids = ai.token_ids(31, shape.vocab, 4, 600)
    force = _half_forced(32, ids.shape, shape.n_layers)
    delta = 0.70
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=640)
    rep = LC.Report(say)
    res, cache, chk = _tf_prefill(model, w, shape, ids, O.ExitConfig(delta=delta),
                                  B.exit_cfg(delta, shape.n_layers, "global"), force=force,
                                  rep=rep)
    rep.summary()
    el = chk.exit_layer
    say(f"  exits {int(np.sum(el < shape.n_layers))} of {el.size} "
        f"(policy {int(np.sum((force.reshape(-1) == 0) & (el < shape.n_layers)))})")
    assert 0 < np.sum(el < shape.n_layers) < el.size
    del model, cache, res
    torch.cuda.empty_cache()


@pytest.mark.parametrize("kv_fused", [True, False])
def test_7b_width_decode_teacher_forced(w7b, kv_fused):
    """Decode at the 7B layer shapes (64 sequences): the skinny stream-K GEMMs
    at their real shapes (ranges straddling column tiles for QKV, gate/up and
    down), key-chunked attention, the deferred KV generation; prompt and
    decode pass checked layer by layer on the GPU's own inputs."""
    shape = SHAPE_7B_4L
    say(f"7B-width decode teacher-forced kv_fused={kv_fused}")
    w32, w = w7b
    N = shape.n_layers
    Bn, T = 64, 2
    ids = ai.token_ids(22, shape.vocab, Bn, T)
    step = ai.token_ids(23, shape.vocab, 1, Bn)[0]
    rng = np.random.default_rng(24)
    force_p = rng.integers(0, N + 1, size=ids.shape).astype(np.int32)
    force_s = rng.integers(1, N + 1, size=Bn).astype(np.int32)
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=64, kv_fused=kv_fused)
    cfg_g = B.exit_cfg(math.inf, N, "global")
    cfg_o = O.ExitConfig(delta=math.inf)
    rep = LC.Report(say)
    _, cache, _ = _tf_prefill(model, w, shape, ids, cfg_o, cfg_g, force=force_p, s_max=T + 1,
                              logits="last", rep=rep)
    _, chk = _tf_decode(model, w, shape, cache, step, np.full(Bn, T), cfg_o, cfg_g,
                        force=force_s, rep=rep)
    rep.summary()
    assert 0 < int(np.sum(chk.exit_layer < N)) < Bn


def test_decode_schedules_agree():
    """The fused and the deferred decode schedules fill the same cache: a
    prompt, then three decode passes with a seeded schedule, run once per
    schedule from the same prompt cache.  After the first pass every cache
    entry is within one bf16 rounding of the other schedule's (the two GEMMs
    sum in different orders); later passes attend to those entries, so after
    the last one the bound is the per-element bf16 bound; exit layers equal,
    logits within 2e-2; the entries no pass wrote stay as the prompt left
    them."""
    say("decode schedules agree")
    shape = SMALL_BF16
    N = shape.n_layers
    w32 = ai.decoder_weights(shape, seed=9, dtype="bf16", std=0.03)
    Bn, T, S = 5, 24, 3
    ids = ai.token_ids(15, shape.vocab, Bn, T)
    step_ids = ai.token_ids(16, shape.vocab, S, Bn)
    rng = np.random.default_rng(17)
    force_s = rng.integers(1, N + 1, size=(S, Bn)).astype(np.int32)
    cfg = B.exit_cfg(math.inf, N, "global")
    outs = []
    base = None
    for fused in (True, False):
        model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=64, kv_fused=fused)
        # slots a pass has not reached yet hold zeros in both runs
        _, cache = model.prefill(ids, cfg, s_max=T + S, logits="last",
                                 cache=model.new_cache(Bn, T + S, fill=0.0))
        if base is None:
            base = (cache.k.clone(), cache.v.clone())
        logits, els, first = [], [], None
        for s in range(S):
            r = model.decode_step(cache, torch.from_numpy(step_ids[s]).to("cuda", torch.int32),
                                  torch.full((Bn,), T + s, dtype=torch.int32, device="cuda"), cfg,
                                  force_layer=torch.from_numpy(force_s[s]).to("cuda", torch.int32),
                                  pos_max=T + s)
            logits.append(r.logits.clone())
            els.append(r.exit_layer.clone())
            if s == 0:
                first = (cache.k.clone(), cache.v.clone())
        torch.cuda.synchronize()
        outs.append((cache, logits, els, first))
    (c1, l1, e1, f1), (c2, l2, e2, f2) = outs
    for a, b in zip(e1, e2):
        assert torch.equal(a, b)
    for a, b in zip(l1, l2):
        assert float((a - b).abs().max()) <= 2e-2
    for a, b in zip(f1, f2):
        a, b = a.float(), b.float()
        ulp = torch.maximum(b.abs(), torch.full_like(b, 2.0 ** -126)) * 2.0 ** -7
        assert bool(((a - b).abs() <= ulp).all())
        assert int((a != b).sum()) <= a.numel() // 100
    for x1, x2, x0 in ((c1.k, c2.k, base[0]), (c1.v, c2.v, base[1])):
        a, b = x1.float(), x2.float()
        assert bool(((a - b).abs() <= torch.clamp(b.abs() * 2.0 ** -7, min=2e-2)).all())
        untouched = torch.ones(N, Bn, T + S, dtype=torch.bool, device=a.device)
        untouched[:, :, T:] = False     # decode slots (written by one schedule or the other)
        u = untouched.reshape(N, Bn * (T + S))
        assert torch.equal(x1[u], x0[u]) and torch.equal(x2[u], x0[u])


def test_timing_select_prefix():
    """adept_timing_select: with a prefix only the matching launches are
    bracketed by events; with none, every launch is again."""
    shape = SMALL_BF16
    w32 = ai.decoder_weights(shape, seed=9, dtype="bf16", std=0.03)
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=512)
    ids = ai.token_ids(14, shape.vocab, 2, 16)
    cfg = B.exit_cfg(math.inf, shape.n_layers, "global")
    res, cache = model.prefill(ids, cfg, s_max=20, logits="last")
    nxt = torch.from_numpy(ids[:, -1].copy()).to("cuda", torch.int32)

    def timed(prefix):
        B.timing_reset()
        B.timing_select(prefix)
        B.timing_enable(True)
        try:
            model.decode_step(cache, nxt, torch.full((2,), 16, dtype=torch.int32, device="cuda"),
                              cfg)
            torch.cuda.synchronize()
        finally:
            B.timing_enable(False)
            B.timing_select(None)
        return B.timing_read()

    only = timed("attend_split")
    assert only and all(k.startswith("attend_split") for k in only), only
    assert only[next(iter(only))][0] == shape.n_layers
    every = timed(None)
    assert set(only) < set(every) and any(k.startswith("gemm_") for k in every), every
