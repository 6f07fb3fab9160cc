"""Compute-reduction accounting of the paper (Section 6, Discussion).

TEST INFRASTRUCTURE ONLY (see adept_oracle).

Two accountings are provided:
  * "paper": multiply-accumulates of the dense projections per token and
    layer (4 D^2 for Q/K/V/O, 2 D F for a two-matrix FFN), the LM head D V
    once per token, and KV generation charged D^2 per skipped layer.  This is
    the only convention under which the GPT2-XL figures of Section 6 (exit
    of every token at layer 38 of 48: 19.7 % saved without KV generation,
    18.1 % with it) are reproduced.
  * "algorithmic": the same, but KV generation charged what the K and V
    projections really cost, 2 D D_q per skipped layer (Eq. 9 uses
    W^{kv} of size D_h x 2 D_q).
Attention-score work, which depends on sequence length, is left out of both,
as the paper's layer costs do.
"""
from __future__ import annotations

import numpy as np


def layer_macs(d_model, d_ff, ffn_mats=2, d_q=None):
    d_q = d_model if d_q is None else d_q
    return 4 * d_model * d_q + ffn_mats * d_model * d_ff


def reduction(n_layers, d_model, d_ff, vocab, exit_layers, kv_accounting="paper",
              ffn_mats=2, d_q=None):
    """Fraction of the full-depth MACs saved when token t exits at
    exit_layers[t] (1-based; n_layers = ran to the end)."""
    d_q = d_model if d_q is None else d_q
    exit_layers = np.asarray(exit_layers)
    per_layer = layer_macs(d_model, d_ff, ffn_mats, d_q)
    full = n_layers * per_layer + d_model * vocab
    skipped = (n_layers - exit_layers).astype(np.float64)
    if kv_accounting == "none":
        kv = 0.0
    elif kv_accounting == "paper":
        kv = float(d_model * d_model)
    elif kv_accounting == "algorithmic":
        kv = float(2 * d_model * d_q)
    else:
        raise ValueError(kv_accounting)
    saved = skipped * (per_layer - kv)
    return float(np.sum(saved) / (exit_layers.size * full))


def exit_module_flops(d_model, vocab):
    """FLOPs of an LM-head-sized exit classifier evaluated at one layer for one
    token (the module-based metric that Section 6 argues against)."""
    return 2 * d_model * vocab


def break_even_layer(n_layers, layer_cost, module_cost):
    """Exit layer before which a per-layer exit module of cost module_cost
    still saves compute: i * (layer + module) < N * layer."""
    return n_layers * layer_cost / (layer_cost + module_cost)
