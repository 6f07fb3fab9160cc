"""Classification mode (Section 4.3) on the GPU against the oracle: a
BERT-style post-norm encoder with token-level exit, where exited tokens
leave the key set and each sequence's [CLS] row at its exit feeds the linear
head.  bf16 throughout, teacher-forced per layer (tests/layer_check.py):
each layer's GPU input goes to the oracle's encoder layer, h within
max(2e-2, one bf16 ulp) per element, decisions / lists / exit layers
bit-exact on identical inputs; free-running decisions end to end are compared
where the oracle's margin exceeds the bf16 error."""
import math
import sys

import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import adept_oracle as O
from paper_2601_03700_amd import binding as B
from paper_2601_03700_amd.model import EncoderModel
from tests import layer_check as LC

pytestmark = pytest.mark.gpu

ENC = ai.EncoderShape(n_layers=4, d_model=256, n_heads=4, head_dim=64, d_ff=512, vocab=300,
                      max_pos=128)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def enc():
    w32 = ai.encoder_weights(ENC, seed=21, dtype="bf16", std=0.05)
    return w32, O.as64(w32), EncoderModel(ENC, w32)


def _tf_classify(model, w, ids, delta, metric="global", force=None, stop_at_cls=True):
    """Classification with the teacher-forced per-layer check: each layer's
    GPU input (the live rows) goes to the oracle's encoder layer; h within
    max(2e-2, one bf16 ulp) per element, exit flags / lists / exit layers
    bit-exact on identical inputs, logits of the GPU's [CLS] states within
    2e-2."""
    rep = LC.Report(say)
    chk = LC.EncoderLayerCheck(w, ENC, O.ExitConfig(delta=delta, metric=metric),
                               force_layer=force, report=rep, stop_at_cls=stop_at_cls)
    out = model.classify(ids, B.exit_cfg(delta, ENC.n_layers, metric), force_layer=force,
                         on_layer=chk, stop_at_cls=stop_at_cls)
    chk.finish(out, ids.shape[1])
    rep.summary()
    return out, chk


@pytest.mark.parametrize("stop_at_cls", [True, False])
@pytest.mark.parametrize("Bn,T", [(3, 100), (2, 24)])   # tiled GEMMs; skinny GEMMs (48 rows)
def test_classify_forced_schedule(enc, Bn, T, stop_at_cls):
    w32, w, model = enc
    say(f"classify forced schedule B={Bn} T={T} stop_at_cls={stop_at_cls}")
    ids = ai.token_ids(30 + T, ENC.vocab, Bn, T)
    force = np.random.default_rng(T).integers(0, ENC.n_layers + 1, size=ids.shape)
    force[0, 0] = 2                       # a [CLS] row that exits early
    out, chk = _tf_classify(model, w, ids, math.inf, force=force, stop_at_cls=stop_at_cls)
    assert int(out.cls_exit_layer[0]) == 2
    el = chk.exit_layer.reshape(Bn, T)
    if stop_at_cls:
        assert (el[0] <= 2).all()


def test_classify_stop_at_cls_same_logits(enc):
    """Stopping a sequence when its [CLS] row exits leaves the logits bit for
    bit as they are without the stop (every kernel computes a row from that
    row's own inputs, and the stop only takes rows out after their [CLS] row
    has left), and leaves fewer rows in the later layers."""
    w32, w, model = enc
    say("classify stop at [CLS]: same logits")
    ids = ai.token_ids(43, ENC.vocab, 3, 80)
    full = O.classify(w, ENC, ids, O.ExitConfig(delta=math.inf))
    fin = np.sort(full.sims[:ENC.n_layers - 1][np.isfinite(full.sims[:ENC.n_layers - 1])])
    q = np.searchsorted(fin, np.quantile(fin, 0.5))
    delta = float(0.5 * (fin[q - 1] + fin[q]))
    cfg = B.exit_cfg(delta, ENC.n_layers, "global")
    go = model.classify(ids, cfg, stop_at_cls=False)
    lg_go, el_go = go.logits.clone(), go.exit_layer.clone()
    st = model.classify(ids, cfg, stop_at_cls=True)
    torch.cuda.synchronize()
    assert torch.equal(st.logits, lg_go)
    el_st, el_go = st.exit_layer.cpu().numpy().reshape(3, 80), el_go.cpu().numpy().reshape(3, 80)
    np.testing.assert_array_equal(el_st, np.minimum(el_go, el_go[:, :1]))
    assert (el_st < el_go).any()


def test_classify_full_depth(enc):
    w32, w, model = enc
    say("classify full depth")
    ids = ai.token_ids(40, ENC.vocab, 2, 128)
    out, _ = _tf_classify(model, w, ids, math.inf)
    assert (out.exit_layer.cpu().numpy() == ENC.n_layers).all()


def test_classify_policy_teacher_forced(enc):
    """The policy at a threshold that fires (global metric), every layer on
    the GPU's own inputs; the other rows keep going after their [CLS] row
    exits, so that later layers still decide."""
    w32, w, model = enc
    say("classify policy teacher-forced")
    ids = ai.token_ids(42, ENC.vocab, 3, 80)
    full = O.classify(w, ENC, ids, O.ExitConfig(delta=math.inf))
    fin = np.sort(full.sims[:ENC.n_layers - 1][np.isfinite(full.sims[:ENC.n_layers - 1])])
    q = np.searchsorted(fin, np.quantile(fin, 0.5))
    delta = float(0.5 * (fin[q - 1] + fin[q]))
    out, chk = _tf_classify(model, w, ids, delta, stop_at_cls=False)
    assert 0 < np.sum(chk.exit_layer < ENC.n_layers) < chk.exit_layer.size


@pytest.mark.parametrize("metric", ["global", "both"])
def test_classify_policy_decisions(enc, metric):
    """A threshold between the oracle's similarities (global or combined
    metric): every token whose margin exceeds 5e-3 at every tested layer exits
    at the same layer on both sides."""
    w32, w, model = enc
    say(f"classify policy metric={metric}")
    ids = ai.token_ids(41, ENC.vocab, 2, 96)
    full = O.classify(w, ENC, ids, O.ExitConfig(delta=math.inf, metric=metric))
    sims = full.sims[:ENC.n_layers - 1]
    fin = np.sort(sims[np.isfinite(sims)])
    q = np.searchsorted(fin, np.quantile(fin, 0.6))
    delta = float(0.5 * (fin[q - 1] + fin[q]))
    ref = O.classify(w, ENC, ids, O.ExitConfig(delta=delta, metric=metric), stop_at_cls=False)
    out = model.classify(ids, B.exit_cfg(delta, ENC.n_layers, metric), stop_at_cls=False)
    torch.cuda.synchronize()
    m = np.abs(ref.sims - delta)
    safe = np.nanmin(np.where(np.isfinite(m), m, np.inf), axis=0) > 5e-3
    el_g, el_o = out.exit_layer.cpu().numpy(), ref.exit_layer
    assert safe.sum() > 0.3 * safe.size
    np.testing.assert_array_equal(el_g[safe], el_o[safe])
    assert 0 < np.sum(el_o < ENC.n_layers) < el_o.size
