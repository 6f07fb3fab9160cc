"""Compute-reduction (RDC) accounting of a run's exit layers (Section 6,
Discussion; the reductions reported in Tables 1 and 3-5).

A token that exits at layer i* skips the dense work of layers i*+1..N and
instead pays for the keys/values of those layers (Eq. 9).  Costs are counted
in multiply-accumulates of the dense projections, as the paper does:

  * a layer: Q, K, V, O (4 D D_q) plus the FFN (ffn_mats D F: 3 for SwiGLU,
    2 for a GELU MLP);
  * a token, once: the LM head (D V);
  * attention-score work (length dependent) is left out, as in the paper's
    per-layer costs.

The K/V of a skipped layer is charged in two ways:

  * ``paper``: D^2 per skipped layer, the charge under which Section 6's
    GPT2-XL example comes out (every token exiting at layer 38 of 48 saves
    19.7 % without KV generation and 18.1 % with it);
  * ``algorithmic``: what the K and V projections cost, 2 D D_q per skipped
    layer (W^{kv} has 2 D_q rows).
"""
from __future__ import annotations

import numpy as np

__all__ = ["dense_layer_macs", "rdc"]


def dense_layer_macs(d_model: int, d_q: int, d_ff: int, ffn_mats: int) -> int:
    """MACs of one token through one layer's dense projections."""
    return 4 * d_model * d_q + ffn_mats * d_model * d_ff


def rdc(exit_layers, n_layers: int, d_model: int, d_q: int, d_ff: int, vocab: int,
        ffn_mats: int = 3) -> dict:
    """Fraction of the full-depth MACs that a run with these exit layers
    (1-based; n_layers = ran to the end) saves, under three charges for the
    generated K/V: none, the paper's, and the algorithmic one."""
    el = np.asarray(exit_layers, dtype=np.int64).ravel()
    if el.size == 0:
        return {"without_kv": 0.0, "paper_kv": 0.0, "algorithmic_kv": 0.0}
    if el.min() < 0 or el.max() > n_layers:
        raise ValueError(f"exit layers outside 0..{n_layers}")
    # skipped (token, layer) pairs from the histogram of exit layers
    counts = np.bincount(el, minlength=n_layers + 1)
    pairs = int(np.dot(counts, n_layers - np.arange(n_layers + 1)))
    layer = dense_layer_macs(d_model, d_q, d_ff, ffn_mats)
    total = el.size * (n_layers * layer + d_model * vocab)
    out = {}
    for name, kv in (("without_kv", 0), ("paper_kv", d_model * d_model),
                     ("algorithmic_kv", 2 * d_model * d_q)):
        out[name] = pairs * (layer - kv) / total
    return out
