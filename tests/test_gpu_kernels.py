"""Per-entry-point parity of the HIP path against the CPU oracle.

Both sides get the same seeded inputs (adept_inputs); the GPU side goes
through the C ABI (binding.py).  Integer outputs (exit flags, compacted
index lists, exit layers) must match bit for bit; floating-point outputs
within the tolerances stated at each assertion.
"""
import math
import sys

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import adept_oracle as O
from paper_2601_03700_amd import binding as B

pytestmark = pytest.mark.gpu
DEV = "cuda"
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(DEV) if dtype is None else t.to(DEV).to(dtype)


def host64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def i32(x):
    return dev(np.asarray(x, np.int32))


def count(n):
    return i32([n])


# ----------------------------------------------------------------------------
# exit test (Section 4.1 Eq. 7-8; Appendix H.3)
# ----------------------------------------------------------------------------

EXIT_CASES = [("bf16", 4096, "global"), ("bf16", 4096, "local"), ("bf16", 768, "global"),
              ("bf16", 1000, "local"), ("f32", 256, "global"), ("f32", 256, "local"),
              ("f32", 1028, "global"), ("bf16", 8192, "global"), ("f32", 4100, "global"),
              ("bf16", 16384, "local")]


@pytest.mark.parametrize("dt,D,metric", EXIT_CASES)
def test_exit_test_matches_oracle(dt, D, metric):
    say(f"exit_test dt={dt} D={D} metric={metric}")
    n_tok, N, layer = 700, 8, 3
    seed = 100 + D
    h = ai.normal(seed, "h", (n_tok, D), dtype=dt)
    # a reference correlated with h so the cosines spread over (0, 1)
    ref = ai.normal(seed, "ref", (n_tok, D), dtype="f32") + 1.5 * h
    if metric == "local":
        ref = ai.to_bf16_values(ref) if dt == "bf16" else ref.astype(np.float32)
    h[5] = 0.0                      # zero row: undefined cosine, never exits
    ref[9] = 0.0                    # empty reference: likewise
    rng = np.random.default_rng(seed)
    active = np.sort(rng.choice(n_tok, 601, replace=False)).astype(np.int32)
    active[:2] = [5, 9]
    active = np.sort(active)
    sims_o = O.cosine(h[active], ref[active])
    srt = np.sort(sims_o[np.isfinite(sims_o)])
    delta = float(0.5 * (srt[len(srt) // 2] + srt[len(srt) // 2 + 1]))  # between two tokens
    force = np.zeros(n_tok, np.int32)
    force[active[10]] = layer        # forced exit at this layer
    force[active[11]] = layer + 1    # forced "not now"
    cfg = B.exit_cfg(delta, N, metric)

    h_d = dev(h, TDT[dt])
    ref_d = dev(ref.astype(np.float32)) if metric == "global" else dev(ref, TDT[dt])
    act_d, n_d = i32(active), count(len(active))
    flag_d = torch.full((len(active) + 8,), 7, dtype=torch.uint8, device=DEV)
    sim_d = torch.full((len(active),), -5.0, dtype=torch.float64, device=DEV)
    B.exit_test(D, layer, cfg, act_d, n_d, len(active), h_d,
                ref_d if metric == "local" else None, ref_d if metric == "global" else None,
                i32(force), flag_d, sim_d)
    torch.cuda.synchronize()

    flags_o = O.exit_decision(sims_o, layer, N, delta, 1)
    f = force[active]
    flags_o = np.where(f > 0, (f == layer) & (layer <= N - 1), flags_o)
    sims_g = sim_d.cpu().numpy()
    assert np.isnan(sims_g[active == 5]).all() and np.isnan(sims_g[active == 9]).all()
    ok = np.isfinite(sims_o)
    np.testing.assert_array_equal(np.isfinite(sims_g), ok)
    # both reduce in fp64: only the summation order differs
    np.testing.assert_allclose(sims_g[ok], sims_o[ok], rtol=0, atol=1e-13)
    # no token within fp64 summation-order noise of the threshold
    assert np.min(np.abs(sims_o[ok] - delta)) > 1e-12
    np.testing.assert_array_equal(flag_d[:len(active)].cpu().numpy().astype(bool), flags_o)
    assert (flag_d[len(active):].cpu().numpy() == 7).all()      # nothing written past the count
    if metric == "global":
        new_o = O.inertia_update(ref[active], h[active])
        new_g = ref_d.cpu().numpy()
        # inertia is stored as float: one float rounding of the fp64 update
        np.testing.assert_allclose(new_g[active], new_o, rtol=2 ** -23, atol=2 ** -40)
        untouched = np.setdiff1d(np.arange(n_tok), active)
        np.testing.assert_array_equal(new_g[untouched], ref.astype(np.float32)[untouched])


@pytest.mark.parametrize("dt,D", [("bf16", 4096), ("bf16", 1000), ("f32", 256), ("f32", 4096)])
def test_exit_test_both_metric_matches_oracle(dt, D):
    """Combined metric: exit iff the global and the local cosine both reach
    delta; sim_out is the smaller cosine; the inertia is updated as for the
    global metric."""
    say(f"exit_test both dt={dt} D={D}")
    n_tok, N, layer = 500, 8, 3
    seed = 300 + D
    h = ai.normal(seed, "h", (n_tok, D), dtype=dt)
    # per-row weights of h in both references, so that the two cosines spread
    # independently and each one alone decides for some rows
    rng = np.random.default_rng(seed)
    wg = rng.uniform(0.3, 3.0, (n_tok, 1))
    wl = rng.uniform(0.3, 3.0, (n_tok, 1))
    inertia = (ai.normal(seed, "ref", (n_tok, D), dtype="f32") + wg * h).astype(np.float32)
    prev = ai.normal(seed, "prev", (n_tok, D), dtype="f32") + wl * h
    prev = ai.to_bf16_values(prev) if dt == "bf16" else prev.astype(np.float32)
    h[5] = 0.0
    inertia[9] = 0.0
    prev[13] = 0.0
    active = np.sort(rng.choice(n_tok, 401, replace=False)).astype(np.int32)
    active[:3] = [5, 9, 13]
    active = np.sort(active)
    sims_o = O.similarity(O.BOTH, h[active], inertia[active], prev[active])
    g_o = O.cosine(h[active], inertia[active])
    l_o = O.cosine(h[active], prev[active])
    srt = np.sort(sims_o[np.isfinite(sims_o)])
    delta = float(0.5 * (srt[len(srt) // 2] + srt[len(srt) // 2 + 1]))
    # the threshold splits the tokens so that each cosine alone decides some
    assert np.sum((g_o >= delta) & ~(l_o >= delta)) > 0 and np.sum((l_o >= delta) & ~(g_o >= delta)) > 0
    cfg = B.exit_cfg(delta, N, "both")
    h_d, in_d, pv_d = dev(h, TDT[dt]), dev(inertia), dev(prev, TDT[dt])
    flag_d = torch.full((len(active) + 8,), 7, dtype=torch.uint8, device=DEV)
    sim_d = torch.full((len(active),), -5.0, dtype=torch.float64, device=DEV)
    B.exit_test(D, layer, cfg, i32(active), count(len(active)), len(active), h_d, pv_d, in_d,
                None, flag_d, sim_d)
    torch.cuda.synchronize()
    flags_o = O.exit_decision(sims_o, layer, N, delta, 1)
    sims_g = sim_d.cpu().numpy()
    ok = np.isfinite(sims_o)
    np.testing.assert_array_equal(np.isfinite(sims_g), ok)
    np.testing.assert_allclose(sims_g[ok], sims_o[ok], rtol=0, atol=1e-13)
    assert np.min(np.abs(g_o[np.isfinite(g_o)] - delta)) > 1e-12
    assert np.min(np.abs(l_o[np.isfinite(l_o)] - delta)) > 1e-12
    np.testing.assert_array_equal(flag_d[:len(active)].cpu().numpy().astype(bool), flags_o)
    assert (flag_d[len(active):].cpu().numpy() == 7).all()
    new_o = O.inertia_update(inertia[active], h[active])
    new_g = in_d.cpu().numpy()
    np.testing.assert_allclose(new_g[active], new_o, rtol=2 ** -23, atol=2 ** -40)
    untouched = np.setdiff1d(np.arange(n_tok), active)
    np.testing.assert_array_equal(new_g[untouched], inertia[untouched])


def test_exit_test_window_and_special_thresholds():
    say("exit_test window")
    D, n, N = 512, 64, 6
    h = ai.normal(5, "h", (n, D), dtype="bf16")
    prev = ai.to_bf16_values(h + 0.01 * ai.normal(5, "p", (n, D)))
    act = i32(np.arange(n))
    for layer, delta, i_min, expect in ((N, -1.0, 1, False), (2, -1.0, 3, False),
                                        (3, -1.0, 3, True), (3, math.inf, 1, False)):
        flag = torch.zeros(n, dtype=torch.uint8, device=DEV)
        B.exit_test(D, layer, B.exit_cfg(delta, N, "local", i_min), act, count(n), n,
                    dev(h, torch.bfloat16), dev(prev, torch.bfloat16), None, None, flag)
        torch.cuda.synchronize()
        assert (flag.cpu().numpy() == int(expect)).all(), (layer, delta, i_min)
    # an empty active list writes nothing
    flag = torch.full((8,), 9, dtype=torch.uint8, device=DEV)
    B.exit_test(D, 2, B.exit_cfg(0.5, N, "local"), act, count(0), n, dev(h, torch.bfloat16),
                dev(prev, torch.bfloat16), None, None, flag)
    torch.cuda.synchronize()
    assert (flag.cpu().numpy() == 9).all()


# ----------------------------------------------------------------------------
# compaction (Appendix I)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("n_tok,n_act,p_exit,slack", [
    (16, 16, 0.5, 0), (5000, 4097, 0.3, 0), (16384, 16384, 0.1, 0), (16384, 9000, 0.0, 0),
    (16384, 9000, 1.0, 0), (300000, 200003, 0.4, 0),
    (300000, 300000, 0.0, 0), (300000, 299999, 1.0, 0),   # multi-pass, no / all exits
    (200000, 200000, 0.3, 0),        # multi-pass over a dense list (whole-line exit layers)
    (70000, 65536, 0.5, 0),          # largest single-workgroup list
    (70000, 65537, 0.5, 0),          # smallest multi-pass list
    (1000, 0, 0.5, 64),              # empty list
    (20000, 777, 0.5, 4000),         # device count below max_active (one workgroup)
    (200000, 70001, 0.5, 40000)])    # device count below max_active (multi-pass)
def test_compact_matches_oracle(n_tok, n_act, p_exit, slack):
    say(f"compact n_tok={n_tok} n_act={n_act} p={p_exit} slack={slack}")
    rng = np.random.default_rng(n_tok + n_act)
    active = np.sort(rng.choice(n_tok, n_act, replace=False)).astype(np.int32)
    flags = (rng.random(n_act) < p_exit).astype(np.uint8)
    layer = 7
    el0 = np.full(n_tok, 32, np.int32)
    # entries past the device count: row 0, flagged to exit -> must be ignored
    max_act = n_act + slack
    act_d, n_d = i32(np.concatenate([active, np.zeros(slack, np.int32)])), count(n_act)
    flag_d = dev(np.concatenate([flags, np.ones(slack, np.uint8), np.zeros(8, np.uint8)]))
    nxt = torch.full((max(n_tok, 1),), -1, dtype=torch.int32, device=DEV)
    ext = torch.full((max(n_tok, 1),), -1, dtype=torch.int32, device=DEV)
    cnt = torch.full((2,), -1, dtype=torch.int32, device=DEV)
    el = i32(el0)
    wsb = B.compact_workspace_bytes(max_act)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=DEV) if wsb else None
    B.compact(layer, 32, flag_d, act_d, n_d, max_act, nxt, cnt[0:1], ext, cnt[1:2], el, ws)
    torch.cuda.synchronize()
    still, gone = O.compact(flags.astype(bool), active)
    c = cnt.cpu().numpy()
    assert c.tolist() == [len(still), len(gone)]
    np.testing.assert_array_equal(nxt.cpu().numpy()[:len(still)], still)
    np.testing.assert_array_equal(ext.cpu().numpy()[:len(gone)], gone)
    assert (nxt.cpu().numpy()[len(still):] == -1).all() and (ext.cpu().numpy()[len(gone):] == -1).all()
    expect = el0.copy()
    expect[gone] = layer
    np.testing.assert_array_equal(el.cpu().numpy(), expect)


def test_compact_worked_example():
    """Appendix I: <am> exits after layer 1, <a> after layer 2: 4 -> 3 -> 2 rows."""
    say("compact worked example")
    act = i32([0, 1, 2, 3])
    n = count(4)
    el = i32([4, 4, 4, 4])
    nxt1, ex1, c1 = (torch.empty(4, dtype=torch.int32, device=DEV) for _ in range(3))
    B.compact(1, 4, dev(np.array([0, 1, 0, 0, 0, 0, 0, 0], np.uint8)), act, n, 4, nxt1, c1[0:1],
              ex1, c1[1:2], el)
    nxt2, ex2, c2 = (torch.empty(4, dtype=torch.int32, device=DEV) for _ in range(3))
    B.compact(2, 4, dev(np.array([0, 1, 0, 0, 0, 0, 0, 0], np.uint8)), nxt1, c1[0:1], 4, nxt2,
              c2[0:1], ex2, c2[1:2], el)
    torch.cuda.synchronize()
    assert int(c1[0]) == 3 and int(c2[0]) == 2
    assert nxt2[:2].cpu().tolist() == [0, 3]
    assert el.cpu().tolist() == [4, 1, 2, 4]


# ----------------------------------------------------------------------------
# decoupled KV generation (Section 4 Eq. 6, Section 4.3 Eq. 9)
# ----------------------------------------------------------------------------

def _kv_case(dt, N, D, H, hd, n_tok, seed, std, exit_lo=0, exit_hi=None):
    shape = ai.DecoderShape(n_layers=N, d_model=D, n_heads=H, head_dim=hd, d_ff=64, vocab=8)
    Dq = H * hd
    s = ai.normal(seed, "s", (n_tok, D), dtype=dt)
    wkv = ai.normal(seed, "wkv", (N, 2 * Dq, D), std=std, dtype=dt)
    gain = ai.gains(seed, "gain", (N, D), dtype=dt)
    exit_hi = N if exit_hi is None else exit_hi
    el = np.random.default_rng(seed).integers(exit_lo, exit_hi + 1, n_tok).astype(np.int32)
    return shape, s, wkv, gain, el


def _layers_for_oracle(wkv, gain, Dq):
    return [{"attn_norm": gain[r], "wk": wkv[r][:Dq], "wv": wkv[r][Dq:]} for r in range(len(gain))]


def _run_kv(dt, shape, s, wkv, gain, el, rows, pos, slot, n_slots, max_pos, fold=True):
    N, D, H, hd = shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim
    Dq = H * hd
    cos = torch.empty((max_pos, hd // 2), dtype=torch.float32, device=DEV)
    sin = torch.empty_like(cos)
    B.rope_table(max_pos, hd, shape.rope_theta, cos, sin)
    kc = torch.full((N, n_slots, H, hd), float("nan"), dtype=TDT[dt], device=DEV)
    vc = torch.full_like(kc, float("nan"))
    wsb = B.kv_generate_workspace_bytes(N, len(rows))
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=DEV)
    w_d, g_d = dev(wkv, TDT[dt]), dev(gain, TDT[dt])
    if fold:
        B.fold_gain(w_d, g_d)   # gains into the columns of [Wk_r; Wv_r]
        g_d = None
    B.kv_generate(N, D, H, hd, shape.rms_eps, dev(s, TDT[dt]), i32(rows), count(len(rows)),
                  len(rows), i32(el), i32(slot), i32(pos), w_d, 2 * Dq * D,
                  g_d, cos, sin, kc, vc, n_slots, ws)
    torch.cuda.synchronize()
    return kc, vc


@pytest.mark.parametrize("dt,hd,fold", [("bf16", 128, True), ("bf16", 64, True),
                                        ("f32", 64, False), ("f32", 64, True)])
def test_kv_generate_matches_oracle(dt, hd, fold):
    say(f"kv_generate dt={dt} hd={hd} fold={fold}")
    N, D, H = 5, 256, 4 if hd == 64 else 2
    n_tok = 300
    shape, s, wkv, gain, el = _kv_case(dt, N, D, H, hd, n_tok, 31 + hd, std=0.0625)
    Dq = H * hd
    rng = np.random.default_rng(3)
    rows = np.sort(rng.choice(n_tok, 257, replace=False)).astype(np.int32)  # ragged tile tail
    pos = rng.integers(0, 2000, n_tok).astype(np.int32)
    slot = rng.permutation(n_tok + 11)[:n_tok].astype(np.int32)
    kc, vc = _run_kv(dt, shape, s, wkv, gain, el, rows, pos, slot, n_tok + 11, 2048, fold)
    _check_kv(dt, shape, s, wkv, gain, el, rows, pos, slot, n_tok + 11, kc, vc)


def _check_kv(dt, shape, s, wkv, gain, el, rows, pos, slot, n_slots, kc, vc):
    N, Dq = shape.n_layers, shape.n_heads * shape.head_dim
    n_tok = n_slots - 11
    gen = O.kv_generate({"layers": _layers_for_oracle(wkv, gain, Dq)}, shape, s[rows], el[rows],
                        pos[rows])
    K, V = host64(kc), host64(vc)
    written = np.zeros((N, n_tok + 11), bool)
    for r, (idx, k, v) in gen.items():
        sl = slot[rows[idx]]
        written[r - 1, sl] = True
        if dt == "f32":
            # fp32: relative to the largest magnitude of the tensor (1e-5)
            for a, b in ((K[r - 1][sl], k), (V[r - 1][sl], v)):
                assert np.max(np.abs(a - b)) <= 1e-5 * np.max(np.abs(b))
        else:
            # bf16: 2e-2 absolute, plus one bf16 ulp of |b| above magnitude 4
            for a, b in ((K[r - 1][sl], k), (V[r - 1][sl], v)):
                tol = np.maximum(2e-2, 2.0 ** (np.floor(np.log2(np.abs(b) + 1e-30)) - 7))
                assert np.all(np.abs(a - b) <= tol), np.max(np.abs(a - b))
    # exactly the (layer, slot) pairs of skipped layers were written
    np.testing.assert_array_equal(~np.isnan(K).any(axis=(2, 3)), written)
    np.testing.assert_array_equal(~np.isnan(V).any(axis=(2, 3)), written)


@pytest.mark.parametrize("D", [64, 128, 192, 320, 448, 512, 576, 704, 1024])
def test_kv_generate_k_depths(D):
    """The GEMM K loop at 1..16 stages of 64: fewer stages than the
    five-slot ring, every remainder of KT mod 5 before the groups of five,
    and the clamped loads past the last stage."""
    say(f"kv_generate K depth D={D}")
    dt, N, H, hd, n_tok = "bf16", 3, 2, 128, 300
    shape, s, wkv, gain, el = _kv_case(dt, N, D, H, hd, n_tok, 500 + D, std=D ** -0.5)
    rng = np.random.default_rng(D)
    rows = np.sort(rng.choice(n_tok, 257, replace=False)).astype(np.int32)
    pos = rng.integers(0, 2000, n_tok).astype(np.int32)
    slot = rng.permutation(n_tok + 11)[:n_tok].astype(np.int32)
    kc, vc = _run_kv(dt, shape, s, wkv, gain, el, rows, pos, slot, n_tok + 11, 2048)
    _check_kv(dt, shape, s, wkv, gain, el, rows, pos, slot, n_tok + 11, kc, vc)


def test_kv_generate_equals_layer_by_layer():
    """Eq. 6: one call over all (token, layer) pairs equals calling once per
    exit layer (each call a separate group) -- decoupling changes nothing."""
    say("kv_generate decoupled vs per-layer")
    dt, N, D, H, hd = "bf16", 6, 256, 2, 128
    shape, s, wkv, gain, el = _kv_case(dt, N, D, H, hd, 200, 77, std=0.0625)
    rows = np.arange(200, dtype=np.int32)
    pos = np.arange(200, dtype=np.int32)
    kc, vc = _run_kv(dt, shape, s, wkv, gain, el, rows, pos, pos, 200, 256)
    for L in range(N):
        sub = rows[el == L]
        if sub.size == 0:
            continue
        k1, v1 = _run_kv(dt, shape, s, wkv, gain, el, sub, pos, pos, 200, 256)
        a = torch.isfinite(k1.float())
        assert torch.equal(k1[a], kc[a]) and torch.equal(v1[a], vc[a])


def test_kv_generate_full_shape_sampled():
    """The standalone KV generation at full shape: 4096 exited tokens of width
    4096, exit layers uniform in 8..31 of a 32-layer stack, per-layer Wk/Wv
    4096 x 4096 N(0, 0.02) with non-unit gains folded in, 32 heads x 128,
    RoPE over positions 0..4095, one call writing a [32][4096][32][128] cache
    (the launch the bench times).  Every slot's written layers are exactly
    i*+1..32 (NaN sentinel); the values of 128 sampled tokens at all of their
    skipped layers match the oracle (Eq. 9) per element within max(2e-2, one
    bf16 ulp)."""
    N, D, H, hd, n = 32, 4096, 32, 128, 4096
    Dq = H * hd
    shape = ai.DecoderShape(n_layers=N, d_model=D, n_heads=H, head_dim=hd, d_ff=64, vocab=8)
    say("kv_generate full shape (4096 tokens, 32 layers, width 4096)")
    g = torch.Generator(device=DEV).manual_seed(11)
    s = torch.randn((n, D), generator=g, device=DEV).to(torch.bfloat16)
    w = torch.empty((N, 2 * Dq, D), dtype=torch.bfloat16, device=DEV)
    for r in range(N):
        w[r].copy_(torch.randn((2 * Dq, D), generator=g, device=DEV).mul_(0.02))
    gain = (1.0 + 0.1 * torch.randn((N, D), generator=g, device=DEV)).to(torch.bfloat16)
    w_fold = w.clone()
    B.fold_gain(w_fold, gain)
    el = ai.forced_exit_layers(12, n, 8, 31)
    rows = torch.arange(n, dtype=torch.int32, device=DEV)
    cos = torch.empty((n, hd // 2), dtype=torch.float32, device=DEV)
    sin = torch.empty_like(cos)
    B.rope_table(n, hd, shape.rope_theta, cos, sin)
    kc = torch.full((N, n, H, hd), float("nan"), dtype=torch.bfloat16, device=DEV)
    vc = torch.full_like(kc, float("nan"))
    ws = torch.empty(B.kv_generate_workspace_bytes(N, n), dtype=torch.uint8, device=DEV)
    B.kv_generate(N, D, H, hd, shape.rms_eps, s, rows, count(n), n, i32(el), rows, rows, w_fold,
                  2 * Dq * D, None, cos, sin, kc, vc, n, ws)
    torch.cuda.synchronize()
    layer = torch.arange(1, N + 1, device=DEV).view(N, 1)
    want = layer > torch.from_numpy(el).to(DEV).view(1, n).long()
    assert torch.equal(~torch.isnan(kc).any(dim=(2, 3)), want)
    assert torch.equal(~torch.isnan(vc).any(dim=(2, 3)), want)
    samp = np.sort(np.random.default_rng(13).choice(n, 128, replace=False))
    samp[0] = int(np.argmin(el))             # an earliest exit: 24 skipped layers

    class Layers:                            # float64 copies of one layer at a time
        def __getitem__(self, r):
            return {"attn_norm": host64(gain[r]), "wk": host64(w[r, :Dq]),
                    "wv": host64(w[r, Dq:])}

    gen = O.kv_generate({"layers": Layers()}, shape, host64(s[samp]), el[samp], samp)
    worst = 0.0
    for r, (idx, k, v) in gen.items():
        sl = torch.from_numpy(samp[idx]).to(DEV)
        for a, b in ((host64(kc[r - 1][sl]), k), (host64(vc[r - 1][sl]), v)):
            tol = np.maximum(2e-2, 2.0 ** (np.floor(np.log2(np.abs(b) + 1e-30)) - 7))
            worst = max(worst, float(np.max(np.abs(a - b) / tol)))
    say(f"  {sum(len(x[0]) for x in gen.values())} sampled (token, layer) pairs, "
        f"worst error {worst:.3f} x the bound")
    assert worst <= 1.0
    del kc, vc, w, w_fold
    torch.cuda.empty_cache()


# ----------------------------------------------------------------------------
# attention over a mixed cache (Section 3 Eq. 5)
# ----------------------------------------------------------------------------

def _attend_case(dt, H, hd, n_seq, s_max, lens, frac_active, seed, causal=True, live=False,
                 decode=False, with_ws=True):
    rng = np.random.default_rng(seed)
    kc = ai.normal(seed, "k", (n_seq * s_max, H, hd), dtype=dt)
    vc = ai.normal(seed, "v", (n_seq * s_max, H, hd), dtype=dt)
    # poison slots past each sequence's length: never read
    for b in range(n_seq):
        kc[b * s_max + lens[b]:(b + 1) * s_max] = np.nan
        vc[b * s_max + lens[b]:(b + 1) * s_max] = np.nan
    if decode:
        rows_pos = np.array(lens) - 1
        pos = rows_pos.astype(np.int32)
        seq = np.arange(n_seq, dtype=np.int32)
        active = np.arange(n_seq, dtype=np.int32)
    else:
        T = s_max
        pos = np.tile(np.arange(T), n_seq).astype(np.int32)
        seq = np.repeat(np.arange(n_seq), T).astype(np.int32)
        cand = np.array([b * T + p for b in range(n_seq) for p in range(lens[b])])
        k = max(1, int(frac_active * cand.size))
        active = np.sort(rng.choice(cand, k, replace=False)).astype(np.int32)
    n = active.size
    q = ai.normal(seed, "q", (n, H, hd), dtype=dt)
    key_live = None
    if live:
        key_live = (rng.random(n_seq * s_max) < 0.7).astype(np.uint8)
        for a in active:  # a live query's own key is live
            key_live[seq[a] * s_max + pos[a]] = 1
    out = torch.full((n + 3, H, hd), 123.0, dtype=TDT[dt], device=DEV)
    ws = None
    if with_ws:
        wsb = B.attend_workspace_bytes(n, n_seq, H, hd, s_max)
        ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    B.attend(H, hd, dev(q, TDT[dt]), i32(active), count(n), n, i32(pos), i32(seq), n_seq,
             dev(kc, TDT[dt]), dev(vc, TDT[dt]), s_max, out, causal=causal,
             key_len=None if causal else i32(lens),
             key_live=None if key_live is None else dev(key_live), workspace=ws)
    torch.cuda.synchronize()
    kc64, vc64 = np.nan_to_num(kc.astype(np.float64)), np.nan_to_num(vc.astype(np.float64))
    km = None
    if key_live is not None:
        km = np.stack([key_live[seq[a] * s_max: seq[a] * s_max + s_max].astype(bool) for a in active])
    ref = O.attend(q.astype(np.float64), kc64, vc64, seq[active] * s_max, pos[active],
                   key_len=np.array(lens)[seq[active]], causal=causal, key_mask=km)
    got = host64(out)
    assert (got[n:] == 123.0).all()
    return got[:n], ref


@pytest.mark.parametrize("hd,H,n_seq,s_max,frac", [(128, 4, 3, 300, 1.0), (128, 4, 2, 1000, 0.37),
                                                   (64, 6, 4, 200, 0.6), (128, 4, 1, 64, 1.0),
                                                   (128, 4, 5, 70, 0.05),
                                                   # heads split evenly over the 8 XCDs:
                                                   # the one-dimensional XCD-major grid
                                                   (128, 8, 3, 300, 0.6), (128, 32, 2, 700, 0.8),
                                                   (64, 16, 3, 257, 1.0), (128, 32, 4, 600, 1.0)])
def test_attend_prefill_mfma_matches_oracle(hd, H, n_seq, s_max, frac):
    say(f"attend prefill hd={hd} H={H} n_seq={n_seq} s_max={s_max} frac={frac}")
    lens = [s_max] * n_seq
    got, ref = _attend_case("bf16", H, hd, n_seq, s_max, lens, frac, 7 + hd + H)
    # bf16 output and bf16 probabilities: 2e-2 absolute on O(1) values
    assert np.max(np.abs(got - ref)) <= 2e-2, np.max(np.abs(got - ref))


@pytest.mark.parametrize("hd,lens,decode,causal,live,H,frac", [
    (128, [1000, 999, 513, 64, 1], True, True, False, 4, 1.0),   # decode, ragged, 1-key sequence
    (64, [700, 255, 256, 257], True, True, False, 6, 1.0),       # decode, chunk-boundary lengths
    (64, [512, 300, 77], False, False, True, 2, 0.01),          # few bidirectional live queries
    (128, [130, 20], False, True, False, 3, 0.02),               # few causal queries per sequence
])
def test_attend_split_matches_oracle(hd, lens, decode, causal, live, H, frac):
    """bf16 key-chunked kernel (fewer than 4 queries per sequence on average)."""
    say(f"attend split hd={hd} lens={lens} decode={decode} causal={causal} live={live}")
    n_seq, s_max = len(lens), max(lens)
    got, ref = _attend_case("bf16", H, hd, n_seq, s_max, lens, frac, 23 + hd, causal=causal,
                            live=live, decode=decode)
    assert np.max(np.abs(got - ref)) <= 2e-2, np.max(np.abs(got - ref))


@pytest.mark.parametrize("hd,lens,live,frac", [(64, [512, 512, 300], True, 0.7),
                                               (64, [100, 512], True, 1.0),
                                               (128, [250, 129, 64], False, 0.5)])
def test_attend_tiles_bidirectional_matches_oracle(hd, lens, live, frac):
    """bf16 query-tile MFMA kernel, bidirectional (classification): every
    query sees all keys of its sequence below key_len, minus the dead ones."""
    say(f"attend tiles bidirectional hd={hd} lens={lens} live={live} frac={frac}")
    n_seq, s_max = len(lens), max(lens)
    got, ref = _attend_case("bf16", 12 if hd == 64 else 4, hd, n_seq, s_max, lens, frac, 31 + hd,
                            causal=False, live=live)
    assert np.max(np.abs(got - ref)) <= 2e-2, np.max(np.abs(got - ref))


@pytest.mark.parametrize("dt,decode,causal,live", [("f32", False, True, False),
                                                   ("f32", True, True, False),
                                                   ("bf16", True, True, False),
                                                   ("bf16", False, False, True),
                                                   ("f32", False, False, True)])
def test_attend_generic_matches_oracle(dt, decode, causal, live):
    say(f"attend generic dt={dt} decode={decode} causal={causal} live={live}")
    n_seq, s_max = 3, 150
    lens = [150, 97, 31] if (decode or not causal) else [150] * 3
    got, ref = _attend_case(dt, 2, 64, n_seq, s_max, lens, 0.5, 11, causal=causal, live=live,
                            decode=decode, with_ws=False)
    if dt == "f32":
        assert np.max(np.abs(got - ref)) <= 1e-5 * np.max(np.abs(ref))
    else:
        assert np.max(np.abs(got - ref)) <= 2e-2


@pytest.mark.parametrize("n_dev", [64, 32, 8, 1])
def test_attend_decode_full_shape_sampled(n_dev):
    """7B-shaped decode attention: 64 sequences, 32 heads x 128, contexts of
    4097..4352 keys (a 4096-token prompt plus up to 256 generated tokens), the
    launch the decode step makes (key chunks + merge).  Caches come from the
    seeded device generator; slots past each context are NaN (never read).
    Sampled (query, head) pairs are checked against the oracle.  n_dev < 64:
    the device count is below the host bound the launch is sized for, so the
    kernels split each context into more chunks (17 at most, one per 256 keys
    of s_max); entries past the count stay untouched."""
    n_seq, H, hd, s_max = 64, 32, 128, 4352
    say(f"attend decode full shape n_seq={n_seq} H={H} hd={hd} s_max={s_max} n_dev={n_dev}")
    g = torch.Generator(device=DEV).manual_seed(41)
    kc = torch.randn((n_seq * s_max, H, hd), generator=g, device=DEV).to(torch.bfloat16)
    vc = torch.randn((n_seq * s_max, H, hd), generator=g, device=DEV).to(torch.bfloat16)
    q = torch.randn((n_seq, H, hd), generator=g, device=DEV).to(torch.bfloat16)
    rng = np.random.default_rng(41)
    lens = rng.integers(4097, s_max + 1, n_seq)
    lens[0], lens[1] = 4097, s_max
    for b in range(n_seq):
        kc[b * s_max + int(lens[b]):(b + 1) * s_max] = float("nan")
        vc[b * s_max + int(lens[b]):(b + 1) * s_max] = float("nan")
    pos = (lens - 1).astype(np.int32)
    seq = np.arange(n_seq, dtype=np.int32)
    out = torch.full((n_seq, H, hd), 123.0, dtype=torch.bfloat16, device=DEV)
    ws = torch.empty(B.attend_workspace_bytes(n_seq, n_seq, H, hd, s_max), dtype=torch.uint8,
                     device=DEV)
    B.attend(H, hd, q, i32(seq), count(n_dev), n_seq, i32(pos), i32(seq), n_seq, kc, vc, s_max,
             out, causal=True, workspace=ws)
    torch.cuda.synchronize()
    got = host64(out)
    assert (got[n_dev:] == 123.0).all()
    got = got[:n_dev]
    assert np.isfinite(got).all()
    # up to 16 sequences (the shortest and longest contexts among them) x 16 heads
    seqs = np.unique(np.concatenate([[0, 1, n_dev - 1],
                                     rng.choice(n_dev, min(13, n_dev), replace=False)]))[:16]
    seqs = seqs[seqs < n_dev]
    worst = 0.0
    for b in seqs:
        L = int(lens[b])
        ks = host64(kc[b * s_max:b * s_max + L])
        vs = host64(vc[b * s_max:b * s_max + L])
        heads = np.unique(np.concatenate([[0, H - 1], rng.choice(H, 14, replace=False)]))
        ref = O.attend(host64(q[b:b + 1]), ks, vs, np.array([0]), np.array([L - 1]))
        err = np.max(np.abs(got[b, heads] - ref[0, heads]))
        worst = max(worst, float(err))
        assert err <= 2e-2, (b, err)
    say(f"  decode attention full shape: max err {worst:.3g} over {len(seqs)} sequences")
    del kc, vc
    torch.cuda.empty_cache()


def test_token_init_beyond_one_grid():
    """adept_token_init with more rows than its capped grid has threads
    (4096 x 256): every row is initialised (grid-stride)."""
    n, N, D = 3 << 19, 32, 8
    say(f"token_init n_tok={n}")
    active = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    el = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(4, dtype=torch.int32, device=DEV)
    inertia = torch.full((n, D), 5.0, dtype=torch.float32, device=DEV)
    B.token_init(n, N, D, active, cnt, el, inertia)
    torch.cuda.synchronize()
    assert int(cnt[0]) == n
    assert torch.equal(active, torch.arange(n, dtype=torch.int32, device=DEV))
    assert bool((el == N).all()) and bool((inertia == 0).all())
