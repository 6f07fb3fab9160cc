"""Pins of the hidden-state-mapper oracle (Section 4.2; Appendix B, Table S1):
library convolution and layers, the paper's parameter counts, and special
weights whose result is known in closed form."""
import json
import os

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import adept_oracle as O
from oracle import hsm as H

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _weights(D, seed=3, std=0.05):
    return H.HSMWeights(**{k: (np.asarray(v, np.float64) if not isinstance(v, float) else v)
                           for k, v in ai.hsm_weights(D, seed, std=std).items()})


def test_param_count_matches_table2():
    g = json.load(open(os.path.join(GOLDEN, "table2_hsm_params.json")))
    for name, row in g["models"].items():
        n = H.n_params(row["d_model"]) / 1e6
        # printed in millions, rounded to the integer the table shows
        assert round(n) == row["printed_millions"], (name, n)


def test_conv_matches_torch_conv2d():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 3, 37))
    k = rng.standard_normal((3, 3))
    want = torch.nn.functional.conv2d(torch.from_numpy(x)[:, None], torch.from_numpy(k)[None, None],
                                      bias=torch.tensor([0.25], dtype=torch.float64),
                                      stride=1, padding=(0, 1))
    np.testing.assert_allclose(H.conv3x3(x, k, 0.25), want[:, 0, 0].numpy(), rtol=0, atol=1e-13)


def test_forward_matches_torch_modules():
    """The same reading of Table S1 assembled from torch layers in fp64."""
    D, n, eps = 32, 7, 1e-6
    w = _weights(D)
    rng = np.random.default_rng(2)
    s, p, i = (rng.standard_normal((n, D)) for _ in range(3))
    f64 = torch.float64
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=f64)
    lin = lambda wt, b: (lambda x: torch.nn.functional.linear(x, t(wt), t(b)))
    rms = lambda g: (lambda x: torch.nn.functional.rms_norm(x, (x.shape[-1],), t(g), eps))
    gelu = torch.nn.GELU(approximate="none")
    x3 = torch.stack([rms(w.g0)(t(s)), rms(w.g0)(t(p)), rms(w.g0)(t(i))], dim=1)[:, None]
    u = torch.nn.functional.conv2d(x3, t(w.conv)[None, None], t([w.conv_b]), padding=(0, 1))[:, 0, 0]
    a = lin(w.w1, w.b1)(u)
    c = lin(w.w3, w.b3)(gelu(lin(w.w2, w.b2)(gelu(a))))
    e = lin(w.w4, w.b4)(rms(w.g1)(c) + a)
    want = rms(w.g2)(e) + u
    np.testing.assert_allclose(H.hsm_forward(w, s, p, i, eps), want.numpy(), rtol=0, atol=1e-12)


def test_special_weights():
    """FC4 = 0 and a conv kernel that picks one stacked state: the output is
    that state's normalised row (plus the conv bias), which fixes the stack
    order (current, previous, inertia) and the padding."""
    D, n, eps = 16, 4, 1e-6
    rng = np.random.default_rng(3)
    s, p, i = (rng.standard_normal((n, D)) for _ in range(3))
    for r, src in enumerate((s, p, i)):
        w = _weights(D)
        w.w4[:] = 0.0
        w.b4[:] = 0.0
        w.conv = np.zeros((3, 3))
        w.conv[r, 1] = 1.0
        w.conv_b = 0.5
        out = H.hsm_forward(w, s, p, i, eps)
        np.testing.assert_allclose(out, O.rms_norm(src, w.g0, eps) + 0.5, rtol=0, atol=1e-13)
    # a shift kernel: column t = 0 reads the left neighbour (zero at d = 0)
    w = _weights(D)
    w.w4[:] = 0.0
    w.b4[:] = 0.0
    w.conv = np.zeros((3, 3))
    w.conv[0, 0] = 1.0
    w.conv_b = 0.0
    out = H.hsm_forward(w, s, p, i, eps)
    x = O.rms_norm(s, w.g0, eps)
    np.testing.assert_allclose(out[:, 1:], x[:, :-1], rtol=0, atol=1e-13)
    np.testing.assert_allclose(out[:, 0], 0.0, atol=1e-15)


SMALL = ai.DecoderShape(n_layers=4, d_model=64, n_heads=4, head_dim=16, d_ff=128, vocab=97)


@pytest.mark.parametrize("metric,forced", [("global", False), ("both", False), ("global", True)])
def test_prefill_with_mapper_equals_token_at_a_time(metric, forced):
    """With the mapper in place of the identity, the batched prefill
    (compaction, decoupled K/V from the mapped state) still equals the
    token-at-a-time recomputation in which each token is mapped at its exit."""
    from oracle import brute_force as BF
    import math
    w = O.as64(ai.decoder_weights(SMALL, seed=11))
    ids = ai.token_ids(12, SMALL.vocab, 2, 12)
    hw = _weights(SMALL.d_model, seed=5, std=0.08)
    mapper = lambda s, p, i: H.hsm_forward(hw, s, p, i, SMALL.rms_eps)
    full, _ = O.prefill(w, SMALL, ids, O.ExitConfig(delta=math.inf, metric=metric))
    sims = full.sims[1:SMALL.n_layers - 1]
    delta = float(np.quantile(sims[np.isfinite(sims)], 0.5))
    cfg = O.ExitConfig(delta=delta, metric=metric)
    force = (np.random.default_rng(4).integers(0, SMALL.n_layers + 1, size=ids.shape)
             if forced else None)
    res, cache = O.prefill(w, SMALL, ids, cfg, force_layer=force, mapper=mapper)
    assert np.sum(res.exit_layer < SMALL.n_layers) > 0
    bf = BF.brute_force_prefill(w, SMALL, ids, cfg, force_layer=force, mapper=mapper)
    B_, T = ids.shape
    for b in range(B_):
        rows = slice(b * T, (b + 1) * T)
        np.testing.assert_array_equal(res.exit_layer[rows], bf[b]["exit_layer"])
        np.testing.assert_allclose(res.logits[rows], bf[b]["logits"], rtol=0, atol=1e-12)
        for r in range(SMALL.n_layers):
            np.testing.assert_allclose(cache.k[r][rows], np.stack(bf[b]["keys"][r]), rtol=0,
                                       atol=1e-12)
    # the mapper changes the result (it is not silently skipped)
    ident, _ = O.prefill(w, SMALL, ids, cfg, force_layer=force)
    assert np.max(np.abs(ident.logits - res.logits)) > 1e-3
