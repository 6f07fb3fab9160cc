"""Host-side compute-reduction accounting of the package against the oracle's
(Section 6, Discussion) and the values the paper prints for its example."""
import json
import os

import numpy as np
import pytest

from oracle import accounting as acc
from paper_2601_03700_amd.accounting import dense_layer_macs, rdc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_rdc_section6_example():
    g = json.load(open(os.path.join(GOLDEN, "section6_accounting.json")))
    x = g["gpt2_xl"]
    r = rdc([g["exit_all_at_layer"]] * 5, x["n_layers"], x["d_model"], x["d_model"], x["d_ff"],
            x["vocab"], ffn_mats=2)
    # printed to one decimal, cut (19.76 -> 19.7)
    assert g["reduction_percent_without_kv_generation"] <= 100 * r["without_kv"] < \
        g["reduction_percent_without_kv_generation"] + 0.1
    assert g["reduction_percent_with_kv_generation"] <= 100 * r["paper_kv"] < \
        g["reduction_percent_with_kv_generation"] + 0.1
    assert r["algorithmic_kv"] < r["paper_kv"] < r["without_kv"]


@pytest.mark.parametrize("shape", [
    (32, 4096, 4096, 11008, 32000, 3),    # Llama-7B-shaped decoder (SwiGLU)
    (48, 1600, 1600, 6400, 50257, 2),     # GPT2-XL shape (two-matrix MLP)
    (12, 768, 768, 3072, 2, 2),           # BERT-base encoder, 2-class head
])
def test_rdc_matches_oracle(shape):
    N, D, Dq, F, V, mats = shape
    rng = np.random.default_rng(7)
    for lo in (1, N // 2, N):
        el = rng.integers(lo, N + 1, size=1000)
        r = rdc(el, N, D, Dq, F, V, ffn_mats=mats)
        for key, kv in (("without_kv", "none"), ("paper_kv", "paper"),
                        ("algorithmic_kv", "algorithmic")):
            want = acc.reduction(N, D, F, V, el, kv, ffn_mats=mats, d_q=Dq)
            assert r[key] == pytest.approx(want, rel=1e-12, abs=1e-15)


def test_rdc_edges():
    assert rdc([], 32, 4096, 4096, 11008, 32000) == \
        {"without_kv": 0.0, "paper_kv": 0.0, "algorithmic_kv": 0.0}
    r = rdc([32] * 7, 32, 4096, 4096, 11008, 32000)
    assert all(v == 0.0 for v in r.values())          # nobody exits: nothing saved
    # every token after layer 0 would skip all layers: the LM head is what is left
    r0 = rdc([0], 4, 8, 8, 16, 10, ffn_mats=3)
    layer = dense_layer_macs(8, 8, 16, 3)
    assert r0["without_kv"] == pytest.approx(4 * layer / (4 * layer + 8 * 10))
    with pytest.raises(ValueError):
        rdc([33], 32, 4096, 4096, 11008, 32000)
