"""Budget-calibrated threshold (paper_2601_03700_amd/calibrate.py) against the
exit rule of Eq. 8 as the oracle states it, on the CPU."""
import math

import numpy as np
import pytest

import adept_inputs as ai
from oracle import adept_oracle as O
from paper_2601_03700_amd import calibrate as C


def brute_skipped(sims, delta, N, i_min):
    """Exit layer of each token by the oracle's rule applied layer by layer
    to fixed similarities, then the skipped (token, layer) fraction."""
    n = sims.shape[1]
    el = np.full(n, N)
    for i in range(1, N + 1):
        flags = O.exit_decision(sims[i - 1], i, N, delta, i_min)
        el = np.where((el == N) & flags, i, el)
    return float(np.sum(N - el)) / (N * n)


def random_sims(seed, N, n):
    rng = np.random.default_rng(seed)
    s = rng.uniform(0.3, 1.0, size=(N, n))
    s[0, : n // 2] = np.nan                 # undefined cosines never exit
    s[rng.random((N, n)) < 0.05] = np.nan
    s[1, 7] = s[N - 2, 7] = s[N - 2, 9] = 0.8125   # ties
    return s


@pytest.mark.parametrize("N,i_min", [(8, 1), (8, 3), (32, 1), (4, 2)])
def test_skipped_fraction_matches_the_exit_rule(N, i_min):
    sims = random_sims(N + i_min, N, 300)
    for delta in (0.3, 0.55, 0.8125, 0.9, 0.99, math.inf, -1.0):
        assert C.skipped_fraction_at(sims, delta, N, i_min) == brute_skipped(sims, delta, N,
                                                                             i_min)


@pytest.mark.parametrize("N,i_min", [(8, 1), (32, 1), (12, 2)])
def test_calibrated_delta_is_the_largest_meeting_the_budget(N, i_min):
    sims = random_sims(7 * N, N, 500)
    cand = np.unique(C.running_max(sims, N, i_min))
    for target in (0.05, 0.10, 0.20, 0.25):
        d = C.calibrate_delta(sims, target, N, i_min)
        assert brute_skipped(sims, d, N, i_min) >= target
        above = cand[cand > d]
        if above.size:      # the next larger threshold misses the budget
            assert brute_skipped(sims, above[0], N, i_min) < target
    assert C.calibrate_delta(sims, 0.0, N, i_min) == math.inf
    with pytest.raises(ValueError):
        C.calibrate_delta(sims, 0.99, N, i_min)


@pytest.mark.parametrize("metric", ["local", "global"])
def test_calibration_realised_exactly_without_interaction(metric):
    """One token per sequence: no token attends to another, so an exit
    changes no other token's similarities and the oracle run at the
    calibrated threshold skips exactly the predicted fraction (>= target)."""
    shape = ai.TINY
    w = O.as64(ai.decoder_weights(shape, seed=1, dtype="f32"))
    ids = ai.token_ids(50, shape.vocab, 40, 1)
    full, _ = O.prefill(w, shape, ids, O.ExitConfig(delta=math.inf, metric=metric))
    for target in (0.1, 0.2, 0.25):
        d = C.calibrate_delta(full.sims, target, shape.n_layers)
        res, _ = O.prefill(w, shape, ids, O.ExitConfig(delta=d, metric=metric))
        got = float(np.sum(shape.n_layers - res.exit_layer)) / (shape.n_layers * ids.size)
        assert got == C.skipped_fraction_at(full.sims, d, shape.n_layers) >= target


def test_calibration_close_with_interaction():
    """A 128-token prompt (tokens attend to earlier ones): the realised
    skipped fraction of the oracle run is near the target."""
    shape = ai.TINY
    w = O.as64(ai.decoder_weights(shape, seed=1, dtype="f32"))
    ids = ai.token_ids(2, shape.vocab, 1, 128)
    full, _ = O.prefill(w, shape, ids, O.ExitConfig(delta=math.inf, metric="local"))
    d = C.calibrate_delta(full.sims, 0.2, shape.n_layers)
    res, _ = O.prefill(w, shape, ids, O.ExitConfig(delta=d, metric="local"))
    got = float(np.sum(shape.n_layers - res.exit_layer)) / (shape.n_layers * ids.size)
    assert abs(got - 0.2) < 0.1
