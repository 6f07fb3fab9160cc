"""Budget-calibrated exit threshold (Section 4.1: delta is chosen so that the
skipped computation meets a budget; the paper's operating points skip 5-25 %
of the token-layers).

Host-side selection of one hyperparameter from the similarities of a pass
that never exits (delta = +inf): it is not a step of the forward pass and
runs once, before the measured passes.

With the exit rule of Eq. 8 (a token exits at the first tested layer
i in [i_min, N-1] whose similarity reaches delta), the number of layers a
token skips at threshold delta is the number of tested layers i whose running
maximum m_i = max(sim_{i_min}, ..., sim_i) reaches delta: m is non-decreasing
in i, so {i : m_i >= delta} = {i*, ..., N-1}, N - i* layers.  The skipped
fraction of a pass is therefore the share of running-maximum values >= delta,
and the largest delta that meets a budget is an order statistic of them.
(In a run with exits the later similarities of the remaining tokens shift a
little, since they attend to generated instead of computed K/V of the exited
tokens, so the realised fraction is close to, not exactly, the target.)
"""
from __future__ import annotations

import math

import numpy as np


def running_max(sims, n_layers, min_exit_layer=1):
    """sims [N, n]: similarity of each token at layers 1..N in a pass without
    exits (NaN where undefined).  Returns [N-1-(i_min-1), n]: the running
    maximum over the tested layers i_min..N-1 (undefined counts as -inf)."""
    s = np.asarray(sims, np.float64)
    lo, hi = max(1, min_exit_layer), n_layers - 1
    if s.shape[0] != n_layers:
        raise ValueError(f"sims has {s.shape[0]} layers, expected {n_layers}")
    if hi < lo:
        return np.full((0, s.shape[1]), -np.inf)
    window = np.where(np.isnan(s[lo - 1:hi]), -np.inf, s[lo - 1:hi])
    return np.maximum.accumulate(window, axis=0)


def skipped_fraction_at(sims, delta, n_layers, min_exit_layer=1):
    """Fraction of the (token, layer) pairs that threshold delta would skip
    in the pass the similarities come from."""
    m = running_max(sims, n_layers, min_exit_layer)
    n = np.asarray(sims).shape[1]
    return float(np.count_nonzero(m >= delta)) / (n_layers * n) if n else 0.0


def calibrate_delta(sims, target_skipped, n_layers, min_exit_layer=1):
    """The largest delta whose skipped fraction on these similarities is at
    least target_skipped (in [0, 1)); +inf for a target of 0.  Raises if no
    threshold reaches the target (it is above what the test window allows)."""
    if not 0.0 <= target_skipped < 1.0:
        raise ValueError("target_skipped must be in [0, 1)")
    if target_skipped == 0.0:
        return math.inf
    m = running_max(sims, n_layers, min_exit_layer).ravel()
    n = np.asarray(sims).shape[1]
    total = n_layers * n
    # pairs to skip; the tolerance keeps e.g. 0.2 * 6000 from rounding up to 1201
    k = max(1, int(math.ceil(target_skipped * total - 1e-9 * total)))
    finite = np.sort(m[np.isfinite(m)])[::-1]
    if k > finite.size:
        raise ValueError(f"at most {finite.size / total:.3f} of the token-layers can "
                         f"be skipped in this window")
    return float(finite[k - 1])


class SimRecorder:
    """on_layer hook of a pass that never exits: keeps each layer's
    similarities (sim_out, aligned with the active list, which is every row
    in order when nothing exits) in a device tensor [N, n_tok] (float64).
    Only a device-to-device copy per layer: nothing is read back."""

    def __init__(self, n_layers, n_tok, device):
        import torch
        self.sims = torch.full((n_layers, n_tok), float("nan"), dtype=torch.float64,
                               device=device)

    def __call__(self, i, st):
        self.sims[i - 1].copy_(st.sim_out[: self.sims.shape[1]])
