"""Teacher-forced, per-layer parity of a GPU token pass against the oracle.

A token pass on the GPU calls a checker after every layer step (the
`on_layer` hook of the host models).  The checker reads back the GPU's own
input to that layer -- the states h_{i-1} of the rows entering it and the
cache entries the layer did not compute itself (K/V generated earlier for
exited tokens) -- and runs the oracle's layer on exactly those inputs, so
bf16 errors do not compound from layer to layer.  Per layer it compares:

  * the exit test (Eq. 7-8): similarities (fp64 on both sides, only the
    summation order differs), decisions bit-exact, the inertia update within
    one float rounding;
  * the active-list update (Appendix I): continuing and exited lists and the
    exit layers, bit-exact;
  * the K/V the layer wrote into the cache for every active row;
  * for sampled rows (all rows when there are few): q, the attention output
    over the mixed computed / generated cache (Eq. 5) and the layer output h_i.

After the pass (`finish`): the K/V generated for exited rows at all of their
skipped layers from the GPU's exit state (Eq. 9) and the logits of the GPU's
final states.

Each kernel is compared on its own inputs as the GPU produced them: q and
the layer's own K/V from the GPU's h_{i-1}; the attention output from the
GPU's q and this layer's cache as the GPU holds it; the layer output from
h_{i-1} and the GPU's attention output.  (The attention's inputs are bf16
values; fed fp64 q and K instead, a peaked softmax turns their rounding into
output differences above 2e-2 that say nothing about the kernel.)

Tolerances, per tensor.  f32 runs: ||a - b||_inf <= 1e-5 ||b||_inf.  bf16
runs: per element |a - b| <= max(2e-2, one bf16 ulp of |b|) (above magnitude
4 a single rounding step of a bf16 value exceeds 2e-2); h is compared as
RMS-normalised rows (the values the next layer consumes: raw h grows with
depth, and its bf16 spacing with it); logits (f32 outputs) within 2e-2.

One stated exception, RESID_ALLOW: a layer rounds its residual stream to
bf16 twice -- the sum after the attention sub-layer (whose rounded value the
FFN sub-layer reads and adds to) and the layer output (the post-norm encoder:
the pre-LayerNorm sum, scaled by the LayerNorm's 1/sigma, then the LayerNorm
output).  Two roundings of up to half an ulp each can reach one full ulp,
which exceeds the bound for values just below a power of two in the
normalised scale; those outputs (h, the encoder's sub-layer outputs, the
mapper's output) are allowed twice the per-element bound, and the measured
worst ratio is reported.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import adept_oracle as O

F32_REL = 1e-5
BF16_ABS = 2e-2
RESID_ALLOW = 2.0     # outputs rounded to bf16 twice (see the module docstring)


def bf16_tol(b):
    """Per-element bound max(2e-2, one bf16 ulp of |b|)."""
    a = np.abs(np.asarray(b, np.float64))
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(a, 2.0 ** -126))) - 7)
    return np.maximum(BF16_ABS, ulp)


def host(t):
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rms_rows(x):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True))


class Report:
    """Largest error of each tensor, and its ratio to the bound (<= 1 passes).
    Violations are collected; summary() prints every tensor and then fails
    if any exceeded its bound."""

    def __init__(self, say=print):
        self.say = say
        self.worst = {}
        self.failed = []

    def check(self, what, a, b, dtype, absolute=False, allow=1.0):
        a = np.asarray(a, np.float64)
        b = np.asarray(b, np.float64)
        assert a.shape == b.shape, (what, a.shape, b.shape)
        if a.size == 0:
            return 0.0
        assert np.isfinite(a).all(), f"{what}: non-finite GPU values"
        err = np.abs(a - b)
        if dtype == "f32" and not absolute:
            ratio = float(err.max() / (F32_REL * max(np.abs(b).max(), 1e-30)))
        elif absolute:
            ratio = float(err.max() / BF16_ABS)
        else:
            ratio = float(np.max(err / bf16_tol(b)))
        if dtype == "f32":
            allow = 1.0
        key = what.split("@")[0]
        prev = self.worst.get(key, (0.0, 0.0, allow))
        self.worst[key] = (max(prev[0], float(err.max())), max(prev[1], ratio), allow)
        if ratio > allow:
            self.failed.append(f"{what}: max err {err.max():.4g}, {ratio:.3f} x the bound "
                               f"(allowed {allow:g})")
        return float(err.max())

    def summary(self):
        for k, (e, r, a) in sorted(self.worst.items()):
            extra = f", allowed {a:g} x" if a != 1.0 else ""
            self.say(f"  {k}: max err {e:.3g} ({r:.2f} x the bound{extra})")
        assert not self.failed, "; ".join(self.failed[:8])


class DecoderLayerCheck:
    """on_layer hook of DecoderModel.token_pass (see the module docstring).

    w: oracle weights (float64 tree); shape: DecoderShape; cache: the GPU
    KVCache of the pass; cfg: oracle ExitConfig of the pass; dtype "f32" or
    "bf16"; force_layer: the pass's teacher-forced exit layers (numpy, or
    None); n_sample: rows per layer whose q / attention / h are compared."""

    def __init__(self, w, shape, cache, cfg, dtype, force_layer=None, n_sample=256, seed=0,
                 report=None, mapper=None):
        if cfg.prompt_level:
            raise NotImplementedError("the all-at-once variant is checked end to end")
        self.w, self.shape, self.cache, self.cfg, self.dt = w, shape, cache, cfg, dtype
        self.force = None if force_layer is None else np.asarray(force_layer).reshape(-1)
        # mapper(h_i, h_{i-1}, inertia before layer i) -> s~ (oracle/hsm.py): the
        # layer step maps the exiting rows in place, so their h_i is not
        # observable; they must then be on the forced schedule, and their
        # mapped state is compared with the oracle mapper applied to the
        # oracle's h_i of the GPU's layer input
        self.mapper = mapper
        self.n_sample = n_sample
        self.rng = np.random.default_rng(seed)
        self.rep = report if report is not None else Report()
        self.exits = 0

    def _cmp(self, what, a, b, absolute=False, allow=1.0):
        return self.rep.check(what, a, b, self.dt, absolute, allow)

    def _sample(self, n):
        if n <= self.n_sample:
            return np.arange(n)
        s = self.rng.choice(n, self.n_sample - 2, replace=False)
        return np.unique(np.concatenate([[0, n - 1], s]))

    def __call__(self, i, st):
        torch.cuda.synchronize()
        sh, cfg = self.shape, self.cfg
        N, H, hd = sh.n_layers, sh.n_heads, sh.head_dim
        if i == 1:
            n = st.n_tok
            self.pos = st.pos.cpu().numpy().astype(np.int64)
            self.seq = st.seq.cpu().numpy().astype(np.int64)
            self.slot = st.slot.cpu().numpy().astype(np.int64)
            self.active = np.arange(n)
            self.exit_layer = np.full(n, N, np.int64)
            self.inertia = np.zeros((n, sh.d_model)) if cfg.metric != O.LOCAL else None
        cnt = st.counts.cpu().numpy()
        n_in, n_out, n_ex = int(cnt[(i - 1) & 1]), int(cnt[i & 1]), int(cnt[2])
        act_t = st.active[(i - 1) & 1][:n_in].long()
        act = act_t.cpu().numpy()
        np.testing.assert_array_equal(act, self.active, err_msg=f"layer {i} active list")
        lw = self.w["layers"][i - 1]
        hp = host(st.h[(i - 1) & 1][act_t])      # the GPU's input h_{i-1}
        hc = host(st.h[i & 1][act_t])            # the GPU's output h_i

        # ---- exit test on identical inputs: fp64 on both sides
        flags_g = st.exit_flag[:n_in].cpu().numpy().astype(bool)
        obs = ~flags_g if self.mapper is not None else np.ones(n_in, bool)   # h_i readable
        inert = self.inertia[act] if self.inertia is not None else None
        inert_pre = None if inert is None else inert.copy()
        sims_o = O.similarity(cfg.metric, hc, inert, hp)
        sims_g = st.sim_out[:n_in].cpu().numpy()
        fin = np.isfinite(sims_o)
        np.testing.assert_array_equal(np.isfinite(sims_g[obs]), fin[obs],
                                      err_msg=f"layer {i} NaN sims")
        if (fin & obs).any():
            assert np.max(np.abs(sims_g[fin & obs] - sims_o[fin & obs])) <= 1e-12, \
                f"layer {i} sims"
        flags_o = O.exit_decision(sims_o, i, N, cfg.delta, cfg.min_exit_layer)
        policy = np.ones(n_in, bool)
        if self.force is not None:
            f = self.force[act]
            policy = f <= 0
            flags_o = np.where(policy, flags_o, (f == i) & (i <= N - 1))
        if self.mapper is not None:
            assert not (policy & ~obs).any(), "with a mapper, exits must be forced"
        if cfg.min_exit_layer <= i <= N - 1:
            # no policy decision within the summation-order noise of delta
            close = policy & fin & obs & (np.abs(sims_o - cfg.delta) <= 1e-11)
            assert not close.any(), f"layer {i}: a similarity within 1e-11 of delta"
        np.testing.assert_array_equal(flags_g, flags_o, err_msg=f"layer {i} exit flags")
        if self.inertia is not None:
            upd_g = host(st.inertia[act_t])
            upd_o = O.inertia_update(self.inertia[act], hc)
            np.testing.assert_allclose(upd_g[obs], upd_o[obs], rtol=2.0 ** -23, atol=2.0 ** -40,
                                       err_msg=f"layer {i} inertia")
            self.inertia[act] = upd_g            # the next layer's input is the GPU's

        # ---- active-list update (Appendix I): bit-exact
        nxt_o, ex_o = O.compact(flags_g, act)
        np.testing.assert_array_equal(st.active[i & 1][:n_out].cpu().numpy(), nxt_o,
                                      err_msg=f"layer {i} continuing rows")
        np.testing.assert_array_equal(st.exited[:n_ex].cpu().numpy(), ex_o,
                                      err_msg=f"layer {i} exited rows")
        self.exit_layer[ex_o] = i
        np.testing.assert_array_equal(st.exit_layer.cpu().numpy(), self.exit_layer,
                                      err_msg=f"layer {i} exit layers")
        self.active = nxt_o
        self.exits += ex_o.size

        if n_in == 0:
            return
        # ---- the regular layer on the GPU's inputs
        pos_a, slot_a = self.pos[act], self.slot[act]
        k_o, v_o = O.layer_kv(lw, hp, pos_a, sh)
        kc = host(self.cache.k[i - 1])
        vc = host(self.cache.v[i - 1])
        self._cmp(f"K (computed)@{i}", kc[slot_a], k_o)
        self._cmp(f"V (computed)@{i}", vc[slot_a], v_o)
        S = self._sample(n_in)
        if self.mapper is not None:
            S = np.union1d(S, np.nonzero(~obs)[0])
        q_o = O.layer_q(lw, sh, hp[S], pos_a[S])
        q_g = host(st.q_buf[:n_in])[S].reshape(-1, H, hd)
        self._cmp(f"q@{i}", q_g, q_o)
        # the attention on its own inputs: the GPU's queries over this layer's
        # cache as the GPU holds it (the layer's own K/V, checked above, and
        # the entries generated at earlier exits, checked in finish())
        o_o = O.attend(q_g, kc, vc, self.seq[act][S] * self.cache.s_max, pos_a[S])
        o_g = host(st.attn_out[:n_in])[S].reshape(-1, H, hd)
        self._cmp(f"attention out@{i}", o_g, o_o)
        # output projection, residual and FFN on their inputs h_{i-1} and o
        h_o = O.layer_out(lw, sh, hp[S], o_g)
        keep = obs[S]
        if self.dt == "f32":
            self._cmp(f"h@{i}", hc[S][keep], h_o[keep])
        else:
            self._cmp(f"h (RMS-normalised)@{i}", rms_rows(hc[S][keep]), rms_rows(h_o[keep]),
                      allow=RESID_ALLOW)
        if self.mapper is not None and (~keep).any():
            m = S[~keep]
            s_o = self.mapper(h_o[~keep], hp[m], inert_pre[m] if inert_pre is not None else None)
            self._cmp(f"mapped state (RMS-normalised)@{i}", rms_rows(hc[m]), rms_rows(s_o),
                      allow=RESID_ALLOW)

    def finish(self, st, logits=None, logit_rows=None, n_gen_sample=256):
        """Generated K/V of exited rows (all their skipped layers) and logits."""
        torch.cuda.synchronize()
        sh = self.shape
        N = sh.n_layers
        el = self.exit_layer
        el_t = torch.from_numpy(el).to(st.h[0].device)
        odd = (el_t & 1).bool().unsqueeze(1)
        h_fin = torch.where(odd, st.h[1], st.h[0])   # each row's state at exit (or after N)
        exited = np.nonzero(el < N)[0]
        if exited.size:
            samp = exited if exited.size <= n_gen_sample else np.sort(
                self.rng.choice(exited, n_gen_sample, replace=False))
            s_map = host(h_fin[torch.from_numpy(samp).to(h_fin.device)])
            gen = O.kv_generate(self.w, sh, s_map, el[samp], self.pos[samp])
            for r, (idx, k, v) in gen.items():
                sl = torch.from_numpy(self.slot[samp[idx]]).to(h_fin.device)
                self._cmp(f"K (generated)@{r}", host(self.cache.k[r - 1][sl]), k)
                self._cmp(f"V (generated)@{r}", host(self.cache.v[r - 1][sl]), v)
        if logits is not None:
            rows = logit_rows.cpu().numpy().astype(np.int64)
            lg_o = O.lm_logits(self.w, sh, host(h_fin[logit_rows.long()]))
            self._cmp("logits", host(logits), lg_o, absolute=self.dt == "bf16")
        return self


class EncoderLayerCheck:
    """on_layer hook of EncoderModel.classify: the oracle encoder layer on the
    GPU's layer input (the live rows of each sequence), then the exit test,
    the active-list update and the exit layers as for the decoder."""

    def __init__(self, w, shape, cfg, force_layer=None, report=None, stop_at_cls=True):
        self.w, self.shape, self.cfg = w, shape, cfg
        self.stop_at_cls = stop_at_cls
        self.force = None if force_layer is None else np.asarray(force_layer).reshape(-1)
        self.rep = report if report is not None else Report()

    def __call__(self, i, st):
        torch.cuda.synchronize()
        sh, cfg = self.shape, self.cfg
        N = sh.n_layers
        if i == 1:
            n = st["n"]
            self.seq = st["seq"].cpu().numpy().astype(np.int64)
            self.active = np.arange(n)
            self.exit_layer = np.full(n, N, np.int64)
            self.inertia = np.zeros((n, sh.d_model)) if cfg.metric != O.LOCAL else None
        cnt = st["counts"].cpu().numpy()
        n_in, n_out, n_ex = int(cnt[(i - 1) & 1]), int(cnt[i & 1]), int(cnt[2])
        act_t = st["active"][(i - 1) & 1][:n_in].long()
        act = act_t.cpu().numpy()
        np.testing.assert_array_equal(act, self.active, err_msg=f"layer {i} active list")
        hp = host(st["h"][(i - 1) & 1][act_t])
        hc = host(st["h"][i & 1][act_t])
        if n_in:
            # each step on the GPU's own input: q/k/v from h_{i-1}, the
            # attention from the GPU's q/k/v, the attention sub-layer output
            # from h_{i-1} and the GPU's attention output, the FFN sub-layer
            # from the GPU's attention sub-layer output
            lw = self.w["layers"][i - 1]
            H, hd = sh.n_heads, sh.head_dim
            q_o, k_o, v_o = O.encoder_qkv(lw, sh, hp)
            q_g = host(st["q_buf"][:n_in]).reshape(n_in, H, hd)
            k_g = host(st["k_buf"][act_t]).reshape(n_in, H, hd)
            v_g = host(st["v_buf"][act_t]).reshape(n_in, H, hd)
            for nm, a, b in (("q", q_g, q_o), ("k", k_g, k_o), ("v", v_g, v_o)):
                self.rep.check(f"{nm}@{i}", a, b, "bf16")
            o_g = host(st["attn_out"][:n_in]).reshape(n_in, H, hd)
            self.rep.check(f"attention out@{i}", o_g,
                           O.encoder_attend(q_g, k_g, v_g, self.seq[act]), "bf16")
            y_g = host(st["y_buf"][act_t])
            self.rep.check(f"attention sub-layer out@{i}", y_g,
                           O.encoder_attention_out(lw, sh, hp, o_g), "bf16", allow=RESID_ALLOW)
            self.rep.check(f"h@{i}", hc, O.encoder_ffn_block(lw, sh, y_g), "bf16",
                           allow=RESID_ALLOW)
        inert = self.inertia[act] if self.inertia is not None else None
        sims_o = O.similarity(cfg.metric, hc, inert, hp)
        sims_g = st["sim_out"][:n_in].cpu().numpy()
        fin = np.isfinite(sims_o)
        np.testing.assert_array_equal(np.isfinite(sims_g), fin)
        if fin.any():
            assert np.max(np.abs(sims_g[fin] - sims_o[fin])) <= 1e-12, f"layer {i} sims"
        flags_o = O.exit_decision(sims_o, i, N, cfg.delta, cfg.min_exit_layer)
        policy = np.ones(n_in, bool)
        if self.force is not None:
            f = self.force[act]
            policy = f <= 0
            flags_o = np.where(policy, flags_o, (f == i) & (i <= N - 1))
        if cfg.min_exit_layer <= i <= N - 1:
            assert not (policy & fin & (np.abs(sims_o - cfg.delta) <= 1e-11)).any()
        if self.stop_at_cls:
            seq_len = st["n"] // (int(self.seq.max()) + 1)
            flags_o = O.cls_stop(flags_o, act, seq_len)
        flags_g = st["exit_flag"][:n_in].cpu().numpy().astype(bool)
        np.testing.assert_array_equal(flags_g, flags_o, err_msg=f"layer {i} exit flags")
        if self.inertia is not None:
            upd_g = host(st["inertia"][act_t])
            np.testing.assert_allclose(upd_g, O.inertia_update(self.inertia[act], hc),
                                       rtol=2.0 ** -23, atol=2.0 ** -40)
            self.inertia[act] = upd_g
        nxt_o, ex_o = O.compact(flags_g, act)
        np.testing.assert_array_equal(st["active"][i & 1][:n_out].cpu().numpy(), nxt_o)
        np.testing.assert_array_equal(st["exited"][:n_ex].cpu().numpy(), ex_o)
        self.exit_layer[ex_o] = i
        np.testing.assert_array_equal(st["exit_layer"].cpu().numpy(), self.exit_layer)
        self.active = nxt_o

    def finish(self, out, seq_len):
        """Logits of the GPU's [CLS] states at their exits (2e-2 absolute)."""
        st = out.state
        el = torch.from_numpy(self.exit_layer).to(st["h"][0].device)
        h_fin = torch.where((el & 1).bool().unsqueeze(1), st["h"][1], st["h"][0])
        cls = torch.arange(0, st["n"], seq_len, device=h_fin.device)
        want = O.classify_logits(self.w, host(h_fin[cls]))
        self.rep.check("logits", host(out.logits), want, "bf16", absolute=True)
        return self
