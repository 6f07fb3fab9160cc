"""Hidden state mapper on the GPU (adept_hsm_forward) against the oracle
(Section 4.2; Appendix B, Table S1)."""
import numpy as np
import pytest
import torch

import adept_inputs as ai
from oracle import hsm as H
from paper_2601_03700_amd import binding as B
from tests import layer_check as LC

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)


def _dev_weights(wn):
    out = {}
    for k, v in wn.items():
        if k in ("conv", "conv_b"):
            out[k] = v
        else:
            out[k] = torch.from_numpy(np.asarray(v, np.float32)).to(DEV).to(torch.bfloat16)
    return out


def close_states(a, b, what):
    """Mapped states are hidden states (s~ replaces h_{i*}): compared as
    RMS-normalised rows, per element within max(2e-2, one bf16 ulp), with
    the allowance of outputs rounded twice (the last norm+add reads the
    bf16-rounded convolution output u and rounds the sum again)."""
    rep = LC.Report(say)
    rep.check(what, LC.rms_rows(a), LC.rms_rows(b), "bf16", allow=LC.RESID_ALLOW)
    rep.summary()


@pytest.mark.parametrize("D,n_tok,n_rows,updated", [(256, 300, 290, 0), (512, 700, 517, 1),
                                                    (256, 40, 1, 1), (1024, 600, 300, 1),
                                                    (2048, 300, 257, 0)])
def test_hsm_forward_matches_oracle(D, n_tok, n_rows, updated):
    say(f"hsm D={D} n_tok={n_tok} rows={n_rows} inertia_updated={updated}")
    eps = 1e-6
    wn = ai.hsm_weights(D, seed=D, dtype="bf16", std=1.0 / np.sqrt(4 * D))
    w64 = H.HSMWeights(**{k: (np.asarray(v, np.float64) if k != "conv_b" else float(v))
                          for k, v in wn.items()})
    h = ai.normal(D, "hsm.h", (n_tok, D), dtype="bf16")
    hp = ai.normal(D, "hsm.hp", (n_tok, D), dtype="bf16")
    # an inertia of three unit states, then (optionally) the update with h
    units = [ai.normal(D, f"hsm.u{j}", (n_tok, D)) for j in range(3)]
    pre = sum(u / np.linalg.norm(u, axis=1, keepdims=True) for u in units).astype(np.float32)
    h64 = h.astype(np.float64)
    post = (pre.astype(np.float64) + h64 / np.linalg.norm(h64, axis=1, keepdims=True)).astype(
        np.float32)
    rng = np.random.default_rng(D + n_rows)
    rows = np.sort(rng.choice(n_tok, n_rows, replace=False)).astype(np.int32)
    want = H.hsm_forward(w64, h64[rows], hp[rows].astype(np.float64),
                         pre[rows].astype(np.float64), eps)

    wd = _dev_weights(wn)
    hw = B.hsm_weights(wd)
    h_d = torch.from_numpy(h).to(DEV).to(torch.bfloat16)
    hp_d = torch.from_numpy(hp).to(DEV).to(torch.bfloat16)
    in_d = torch.from_numpy(post if updated else pre).to(DEV)
    rows_d = torch.from_numpy(rows).to(DEV)
    cnt = torch.tensor([n_rows], dtype=torch.int32, device=DEV)
    max_rows = n_rows + 5
    ws = torch.empty(B.hsm_workspace_bytes(D, max_rows), dtype=torch.uint8, device=DEV)
    out = torch.full((n_tok, D), 7.0, dtype=torch.bfloat16, device=DEV)
    B.hsm_forward(D, eps, hw, rows_d, cnt, max_rows, h_d, hp_d, in_d, updated, out, ws)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    close_states(got[rows], want, "mapped states")
    others = np.setdiff1d(np.arange(n_tok), rows)
    assert (got[others] == 7.0).all()                  # only the listed rows are written
    # in place: the mapped states replace the current states of the listed rows
    B.hsm_forward(D, eps, hw, rows_d, cnt, max_rows, h_d, hp_d, in_d, updated, h_d, ws)
    torch.cuda.synchronize()
    got2 = h_d.float().cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(got2[rows], got[rows])
    np.testing.assert_array_equal(got2[others], h[others])


def test_hsm_forward_empty_and_errors():
    say("hsm empty / errors")
    D = 256
    wd = _dev_weights(ai.hsm_weights(D, seed=1, dtype="bf16"))
    hw = B.hsm_weights(wd)
    h = torch.zeros((8, D), dtype=torch.bfloat16, device=DEV)
    inertia = torch.zeros((8, D), dtype=torch.float32, device=DEV)
    rows = torch.arange(8, dtype=torch.int32, device=DEV)
    zero = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(B.hsm_workspace_bytes(D, 8), dtype=torch.uint8, device=DEV)
    out = torch.full((8, D), 3.0, dtype=torch.bfloat16, device=DEV)
    B.hsm_forward(D, 1e-6, hw, rows, zero, 8, h, h, inertia, 0, out, ws)   # no rows: nothing
    torch.cuda.synchronize()
    assert (out == 3.0).all()
    with pytest.raises(B.AdeptError):
        B.hsm_forward(D, 1e-6, hw, rows, zero, 8, h, h, inertia, 0, out, ws[:100])
    with pytest.raises(B.AdeptError):
        B.hsm_forward(200, 1e-6, hw, rows, zero, 8, h, h, inertia, 0, out, ws)


SMALL_BF16 = ai.DecoderShape(n_layers=6, d_model=512, n_heads=4, head_dim=128, d_ff=1024,
                             vocab=512)


@pytest.mark.parametrize("metric", ["global", "both"])
def test_prefill_with_mapper_teacher_forced(metric):
    """The layer step maps the rows exiting at each layer in place before
    their K/V are generated.  Seeded exit schedule; each layer is checked on
    the GPU's own inputs (tests/layer_check.py), the mapped states against
    the oracle mapper applied to the oracle layer's output, then the K/V
    generated from the GPU's mapped states and the logits."""
    import math
    from oracle import adept_oracle as O
    from paper_2601_03700_amd.model import DecoderModel
    say(f"prefill with mapper, metric={metric}")
    shape = SMALL_BF16
    D = shape.d_model
    w32 = ai.decoder_weights(shape, seed=9, dtype="bf16", std=0.03)
    w = O.as64(w32)
    hn = ai.hsm_weights(D, seed=2, dtype="bf16", std=1.0 / np.sqrt(4 * D))
    h64 = H.HSMWeights(**{k: (np.asarray(v, np.float64) if k != "conv_b" else float(v))
                          for k, v in hn.items()})
    ids = ai.token_ids(10, shape.vocab, 3, 200)
    force = np.random.default_rng(5).integers(0, shape.n_layers + 1, size=ids.shape)
    model = DecoderModel(shape, w32, dtype="bf16", rope_max_pos=512, hsm_weights=hn)
    mapper = lambda s, p, i: H.hsm_forward(h64, s, p, i, shape.rms_eps)
    rep = LC.Report(say)
    cache = model.new_cache(3, 200)
    chk = LC.DecoderLayerCheck(w, shape, cache, O.ExitConfig(delta=math.inf, metric=metric),
                               "bf16", force_layer=force, report=rep, mapper=mapper)
    res_g, _ = model.prefill(ids, B.exit_cfg(math.inf, shape.n_layers, metric),
                             force_layer=force, logits="all", cache=cache, on_layer=chk)
    chk.finish(res_g.state, res_g.logits, res_g.rows)
    rep.summary()
    assert "mapped state (RMS-normalised)" in rep.worst
