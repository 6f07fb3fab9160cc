"""Token-at-a-time recomputation of the early-exit prefill (fp64).

TEST INFRASTRUCTURE ONLY (see adept_oracle).  This is a second, independent
way to compute what the batched prefill with compaction computes, used only
to pin the oracle on tiny inputs.

It follows the sequential reading of the method: tokens are processed one
at a time in position order, each one alone through its own layers, with no
index lists, no slot-addressed cache and no batching.  Every layer keeps a
plain Python list of the key/value vectors of the tokens before the current
one.  When a token exits at layer i*, its keys/values for each skipped layer
r > i* are projected from its exit state (Section 4.3, Eq. 9) and appended
to layer r's list; otherwise the token's own layer computes them.  Because
attention is causal, the batched prefill must reproduce exactly this
(Section 3, Eq. 5 and Section 4, Eq. 6).

Shared primitives (norm, rotary, activation, cosine, decision, inertia
update) come from adept_oracle and are pinned there against library
implementations and closed forms; the layer loop, attention, KV generation
and bookkeeping below are written independently.
"""
from __future__ import annotations

import math

import numpy as np

from .adept_oracle import (BOTH, F64, GLOBAL, apply_rope, cosine, exit_decision, inertia_update,
                           rms_norm, silu)


def _proj_kv(lw, shape, x, p):
    u = rms_norm(x[None, :], lw["attn_norm"], shape.rms_eps)[0]
    k = (lw["wk"] @ u).reshape(1, shape.n_heads, shape.head_dim)
    v = (lw["wv"] @ u).reshape(shape.n_heads, shape.head_dim)
    return apply_rope(k, np.array([p]), shape.rope_theta)[0], v


def brute_force_sequence(weights, shape, ids_row, cfg, force_row=None, prior=None, mapper=None):
    """Process one sequence token by token.

    ids_row: [T] token ids.  prior: optional (keys, values) lists per layer
    from earlier tokens of the same sequence (used to continue a sequence).
    Returns dict with logits [T, V], exit_layer [T], keys/values per layer
    (lists of [H, hd]) and the final states [T, D].
    """
    N, H, hd = shape.n_layers, shape.n_heads, shape.head_dim
    W = weights["layers"]
    keys = [list(prior[0][r]) for r in range(N)] if prior else [[] for _ in range(N)]
    vals = [list(prior[1][r]) for r in range(N)] if prior else [[] for _ in range(N)]
    start = len(keys[0])
    T = len(ids_row)
    logits, exits, finals = [], [], []
    for t in range(T):
        p = start + t
        x = np.asarray(weights["embed"], F64)[int(ids_row[t])].copy()
        inertia = np.zeros_like(x)
        exit_at = N
        for i in range(1, N + 1):
            lw = W[i - 1]
            u = rms_norm(x[None, :], lw["attn_norm"], shape.rms_eps)[0]
            q = apply_rope((lw["wq"] @ u).reshape(1, H, hd), np.array([p]), shape.rope_theta)[0]
            k, v = _proj_kv(lw, shape, x, p)
            keys[i - 1].append(k)
            vals[i - 1].append(v)
            Kl = np.stack(keys[i - 1])          # [p+1, H, hd]: every token so far
            Vl = np.stack(vals[i - 1])
            o = np.zeros((H, hd))
            for hh in range(H):
                sc = Kl[:, hh, :] @ q[hh] / math.sqrt(hd)
                w = np.exp(sc - sc.max())
                w /= w.sum()
                o[hh] = w @ Vl[:, hh, :]
            x1 = x + lw["wo"] @ o.reshape(-1)
            u2 = rms_norm(x1[None, :], lw["ffn_norm"], shape.rms_eps)[0]
            x_new = x1 + lw["w_down"] @ (silu(lw["w_gate"] @ u2) * (lw["w_up"] @ u2))
            if cfg.metric == BOTH:
                # both cosines must pass: two separate decisions, and-ed
                flag = bool(exit_decision(cosine(x_new[None, :], inertia[None, :]), i, N,
                                          cfg.delta, cfg.min_exit_layer)[0]) and \
                    bool(exit_decision(cosine(x_new[None, :], x[None, :]), i, N, cfg.delta,
                                       cfg.min_exit_layer)[0])
            else:
                ref = inertia if cfg.metric == GLOBAL else x
                sim = cosine(x_new[None, :], ref[None, :])
                flag = bool(exit_decision(sim, i, N, cfg.delta, cfg.min_exit_layer)[0])
            if force_row is not None and force_row[t] > 0:
                flag = (force_row[t] == i) and i <= N - 1
            inertia_seen = inertia
            if cfg.metric in (GLOBAL, BOTH):
                inertia = inertia_update(inertia[None, :], x_new[None, :])[0]
            x_prev, x = x, x_new
            if flag:
                exit_at = i
                if mapper is not None and i < N:
                    x = mapper(x[None, :], x_prev[None, :], inertia_seen[None, :])[0]
                for r in range(i + 1, N + 1):
                    kr, vr = _proj_kv(W[r - 1], shape, x, p)
                    keys[r - 1].append(kr)
                    vals[r - 1].append(vr)
                break
        finals.append(x)
        exits.append(exit_at)
        logits.append(weights["lm_head"] @ rms_norm(x[None, :], weights["final_norm"],
                                                    shape.rms_eps)[0])
    return {"logits": np.stack(logits), "exit_layer": np.array(exits), "keys": keys,
            "values": vals, "h_final": np.stack(finals)}


def brute_force_prefill(weights, shape, ids, cfg, force_layer=None, mapper=None):
    """Brute force over a [B, T] batch: sequences are independent."""
    ids = np.asarray(ids)
    outs = []
    for b in range(ids.shape[0]):
        fr = None if force_layer is None else np.asarray(force_layer)[b]
        outs.append(brute_force_sequence(weights, shape, ids[b], cfg, fr, mapper=mapper))
    return outs
