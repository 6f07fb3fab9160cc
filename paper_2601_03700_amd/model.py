"""Host-side driver of the early-exit decoder: device buffers and the layer loop.

Everything numeric runs in libadept (binding.py); this module only owns
device memory (torch tensors), lays out the per-token bookkeeping (positions,
sequence ids, cache slots) and calls the C ABI in order:

    adept_embed -> adept_token_init -> adept_layer_step(i), i = 1..N
                -> adept_final_logits [-> adept_argmax]

(the LayerNorm family: adept_embed_positions and adept_final_logits_layernorm
in place of the embedding gather and the RMSNorm head).

A prefill runs the rows of a [B, T] prompt batch (row b*T + p); a decode
step runs one new token per sequence against the cache the prefill (and
earlier steps) filled, with generated entries for every skipped layer.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math

import numpy as np
import torch

from . import binding as B

_TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclasses.dataclass
class KVCache:
    k: torch.Tensor       # [N, n_seq * s_max, H, hd]
    v: torch.Tensor
    n_seq: int
    s_max: int

    @property
    def n_slots(self):
        return self.n_seq * self.s_max


@dataclasses.dataclass
class PassState:
    """Device buffers of one token pass (prefill batch or decode step)."""
    n_tok: int
    h: list                # two [n_tok, D] buffers (ping-pong)
    inertia: torch.Tensor  # [n_tok, D] f32
    pos: torch.Tensor
    seq: torch.Tensor
    slot: torch.Tensor
    active: list           # two [n_tok] int32
    counts: torch.Tensor   # int32 [4]: n_active[0], n_active[1], n_exited, spare
    exited: torch.Tensor
    exit_layer: torch.Tensor
    exit_flag: torch.Tensor
    sim_out: torch.Tensor
    force_layer: torch.Tensor | None
    q_buf: torch.Tensor
    attn_out: torch.Tensor
    ffn_act: torch.Tensor
    workspace: torch.Tensor | None = None

    def final_h(self, row):
        """[D] final state of a row (state at exit, or after the last layer)."""
        el = int(self.exit_layer[row])
        return self.h[el & 1][row]


@dataclasses.dataclass
class PassResult:
    logits: torch.Tensor       # [n_rows, V] f32 for the requested rows
    rows: torch.Tensor         # token rows of the logits
    exit_layer: torch.Tensor   # [n_tok]
    state: PassState


class DecoderModel:
    """A pre-norm decoder held on the device in the library's layout.

    shape.family "llama": weights like adept_inputs.decoder_weights() (numpy,
    per layer) or adept_inputs.decoder_weights_torch() (stacked torch tensors
    on device).  "gpt2": like adept_inputs.gpt2_weights() or
    gpt2_weights_torch(); the LayerNorm gains and shifts are folded into the
    projections that follow them (w_qkv / b_qkv, w_fc / b_fc) and the LM
    head is the token embedding.
    """

    def __init__(self, shape, weights, dtype="bf16", device="cuda", rope_max_pos=4096,
                 hsm_weights=None, kv_fused=True):
        self.shape = shape
        # decode passes in bf16: exited rows' K/V from the later layers' QKV
        # GEMMs (True) or one grouped generation after the last layer (False)
        self.kv_fused = kv_fused
        self.dtype = dtype
        self.tdt = _TORCH_DT[dtype]
        self.device = torch.device(device)
        self.gpt2 = getattr(shape, "family", "llama") == "gpt2"
        N, D, Dq, F = shape.n_layers, shape.d_model, shape.d_q, shape.d_ff
        dev, tdt = self.device, self.tdt

        def up(x):
            if isinstance(x, torch.Tensor):
                return x.to(dev, tdt).contiguous()
            return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev).to(tdt)

        self.hsm, self._hsm_struct = None, None
        if self.gpt2:
            if dtype != "bf16" or hsm_weights is not None:
                raise ValueError("the LayerNorm family runs in bf16 without a mapper")
            self._init_gpt2(weights, up)
            return
        self.b_qkv = self.b_o = self.b_fc = self.b_proj = None
        if isinstance(weights.get("layers"), list):
            L = weights["layers"]
            stack = lambda k: up(np.stack([lw[k] for lw in L]))
            self.attn_norm, self.ffn_norm = stack("attn_norm"), stack("ffn_norm")
            self.w_qkv = up(np.stack([np.concatenate([lw["wq"], lw["wk"], lw["wv"]]) for lw in L]))
            self.w_o = stack("wo")
            self.w_gate, self.w_up, self.w_down = stack("w_gate"), stack("w_up"), stack("w_down")
        else:
            self.attn_norm, self.ffn_norm = up(weights["attn_norm"]), up(weights["ffn_norm"])
            self.w_qkv = torch.empty((N, 3 * Dq, D), dtype=tdt, device=dev)
            self.w_qkv[:, :Dq].copy_(weights["wq"])
            self.w_qkv[:, Dq:2 * Dq].copy_(weights["wk"])
            self.w_qkv[:, 2 * Dq:].copy_(weights["wv"])
            self.w_o = up(weights["wo"])
            self.w_gate, self.w_up, self.w_down = (up(weights["w_gate"]), up(weights["w_up"]),
                                                   up(weights["w_down"]))
        self.embed = up(weights["embed"])
        self.final_norm = up(weights["final_norm"])
        self.lm_head = up(weights["lm_head"])
        assert self.w_qkv.shape == (N, 3 * Dq, D) and self.w_down.shape == (N, D, F)
        # fold the pre-norm gains into the projections that consume the normalised
        # state (the library applies only the 1/rms row factor)
        B.fold_gain(self.w_qkv, self.attn_norm)
        B.fold_gain(self.w_gate, self.ffn_norm)
        B.fold_gain(self.w_up, self.ffn_norm)
        # optional hidden state mapper (Section 4.2) of the exiting rows: a dict
        # like adept_inputs.hsm_weights(); None keeps the identity mapper
        if hsm_weights is not None:
            self.hsm = {k: (v if k in ("conv", "conv_b") else up(v)) for k, v in hsm_weights.items()}
            self._hsm_struct = B.hsm_weights(self.hsm)
        self.rope_max_pos = rope_max_pos
        half = shape.head_dim // 2
        self.rope_cos = torch.empty((rope_max_pos, half), dtype=torch.float32, device=dev)
        self.rope_sin = torch.empty_like(self.rope_cos)
        B.rope_table(rope_max_pos, shape.head_dim, shape.rope_theta, self.rope_cos, self.rope_sin)

    def _init_gpt2(self, weights, up):
        s = self.shape
        N, D, Dq, F = s.n_layers, s.d_model, s.d_q, s.d_ff
        if isinstance(weights.get("layers"), list):
            L = weights["layers"]
            stack = lambda k: up(np.stack([lw[k] for lw in L]))
            cat = lambda ks: up(np.stack([np.concatenate([lw[k] for k in ks]) for lw in L]))
            ln1_g, ln1_b, ln2_g, ln2_b = (stack("ln1_g"), stack("ln1_b"), stack("ln2_g"),
                                          stack("ln2_b"))
            self.w_qkv, self.b_qkv = cat(("wq", "wk", "wv")), cat(("bq", "bk", "bv"))
            self.w_o, self.b_o = stack("wo"), stack("bo")
            self.w_gate, self.b_fc = stack("w_fc"), stack("b_fc")
            self.w_down, self.b_proj = stack("w_proj"), stack("b_proj")
        else:
            ln1_g, ln1_b = up(weights["ln1_g"]), up(weights["ln1_b"])
            ln2_g, ln2_b = up(weights["ln2_g"]), up(weights["ln2_b"])
            self.w_qkv = torch.cat([up(weights[k]) for k in ("wq", "wk", "wv")], 1).contiguous()
            self.b_qkv = torch.cat([up(weights[k]) for k in ("bq", "bk", "bv")], 1).contiguous()
            self.w_o, self.b_o = up(weights["wo"]), up(weights["bo"])
            self.w_gate, self.b_fc = up(weights["w_fc"]), up(weights["b_fc"])
            self.w_down, self.b_proj = up(weights["w_proj"]), up(weights["b_proj"])
        self.w_up = None
        self.embed, self.pos_embed = up(weights["embed"]), up(weights["pos_embed"])
        self.final_ln_g, self.final_ln_b = up(weights["final_ln_g"]), up(weights["final_ln_b"])
        self.lm_head = self.embed      # tied
        assert self.w_qkv.shape == (N, 3 * Dq, D) and self.b_qkv.shape == (N, 3 * Dq)
        assert self.w_down.shape == (N, D, F) and self.pos_embed.shape == (s.max_pos, D)
        # LayerNorm shift into the bias (on the unfolded weights), then the
        # gain into the weights: LN(x) W^T + b = xh (W diag g)^T + (b + W beta)
        B.fold_bias(self.w_qkv, ln1_b, self.b_qkv)
        B.fold_gain(self.w_qkv, ln1_g)
        B.fold_bias(self.w_gate, ln2_b, self.b_fc)
        B.fold_gain(self.w_gate, ln2_g)
        self.rope_cos = self.rope_sin = None
        self.rope_max_pos = s.max_pos     # the position table bounds the positions

    # ------------------------------------------------------------------ buffers
    def new_cache(self, n_seq, s_max, fill=None):
        s = self.shape
        dims = (s.n_layers, n_seq * s_max, s.n_heads, s.head_dim)
        if fill is None:
            k = torch.empty(dims, dtype=self.tdt, device=self.device)
            v = torch.empty(dims, dtype=self.tdt, device=self.device)
        else:
            k = torch.full(dims, fill, dtype=self.tdt, device=self.device)
            v = torch.full(dims, fill, dtype=self.tdt, device=self.device)
        return KVCache(k, v, n_seq, s_max)

    def new_state(self, n_tok, pos, seq, slot, force_layer=None):
        s, dev, tdt = self.shape, self.device, self.tdt
        i32 = dict(dtype=torch.int32, device=dev)
        st = PassState(
            n_tok=n_tok,
            h=[torch.empty((n_tok, s.d_model), dtype=tdt, device=dev) for _ in range(2)],
            inertia=torch.empty((n_tok, s.d_model), dtype=torch.float32, device=dev),
            pos=pos, seq=seq, slot=slot,
            active=[torch.empty(n_tok, **i32) for _ in range(2)],
            counts=torch.zeros(4, **i32),
            exited=torch.empty(n_tok, **i32),
            exit_layer=torch.empty(n_tok, **i32),
            exit_flag=torch.empty(max(n_tok, 4), dtype=torch.uint8, device=dev),
            sim_out=torch.empty(n_tok, dtype=torch.float64, device=dev),
            force_layer=force_layer,
            q_buf=torch.empty((n_tok, s.d_q), dtype=tdt, device=dev),
            attn_out=torch.empty((n_tok, s.d_q), dtype=tdt, device=dev),
            ffn_act=torch.empty((n_tok, s.d_ff), dtype=tdt, device=dev),
        )
        return st

    def layer_args(self, st, cache, cfg, attn_tiles):
        s = self.shape
        a = B.LayerArgs()
        a.dtype = B.dtype_code(self.dtype)
        a.n_layers, a.d_model, a.n_heads = s.n_layers, s.d_model, s.n_heads
        a.head_dim, a.d_ff = s.head_dim, s.d_ff
        a.rms_eps = s.ln_eps if self.gpt2 else s.rms_eps
        a.exit = cfg
        a.w_qkv, a.w_o, a.w_gate = B.ptr(self.w_qkv), B.ptr(self.w_o), B.ptr(self.w_gate)
        a.w_up, a.w_down = B.ptr(self.w_up), B.ptr(self.w_down)
        a.rope_cos, a.rope_sin, a.rope_max_pos = B.ptr(self.rope_cos), B.ptr(self.rope_sin), self.rope_max_pos
        a.family = B.FAMILY_GPT2 if self.gpt2 else B.FAMILY_LLAMA
        a.b_qkv, a.b_o = B.ptr(self.b_qkv), B.ptr(self.b_o)
        a.b_fc, a.b_proj = B.ptr(self.b_fc), B.ptr(self.b_proj)
        a.n_tok, a.max_active, a.n_seq, a.s_max = st.n_tok, st.n_tok, cache.n_seq, cache.s_max
        a.attn_tiles = int(attn_tiles)
        a.kv_fused = int(bool(self.kv_fused) and not attn_tiles and self.dtype == "bf16")
        a.h[0], a.h[1] = B.ptr(st.h[0]), B.ptr(st.h[1])
        a.inertia, a.pos, a.seq, a.slot = B.ptr(st.inertia), B.ptr(st.pos), B.ptr(st.seq), B.ptr(st.slot)
        a.active[0], a.active[1] = B.ptr(st.active[0]), B.ptr(st.active[1])
        cp = B.ptr(st.counts)
        a.n_active[0], a.n_active[1], a.n_exited = cp, cp + 4, cp + 8
        a.exited, a.exit_layer, a.exit_flag = B.ptr(st.exited), B.ptr(st.exit_layer), B.ptr(st.exit_flag)
        a.sim_out = B.ptr(st.sim_out)
        a.force_layer = B.ptr(st.force_layer)
        a.k_cache, a.v_cache, a.n_slots = B.ptr(cache.k), B.ptr(cache.v), cache.n_slots
        a.q_buf, a.attn_out, a.ffn_act = B.ptr(st.q_buf), B.ptr(st.attn_out), B.ptr(st.ffn_act)
        a.hsm = ctypes.addressof(self._hsm_struct) if self._hsm_struct is not None else None
        need = B.layer_workspace_bytes(a)
        if st.workspace is None or st.workspace.numel() < need:
            st.workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        a.workspace, a.workspace_bytes = B.ptr(st.workspace), st.workspace.numel()
        return a

    # ------------------------------------------------------------------ passes
    def _check_positions(self, pos, s_max, pos_max=None):
        """Positions must lie inside the rotary (or position) table and the cache; pos_max
        (a host int, when the caller knows it) avoids reading pos back."""
        pmax = pos_max if pos_max is not None else (int(pos.max()) if pos.numel() else 0)
        if pmax >= self.rope_max_pos or pmax >= s_max:
            raise ValueError(f"position {pmax} outside rotary table / cache")

    def token_pass(self, ids, pos, seq, cache, cfg, force_layer=None, attn_tiles=True,
                   logit_rows=None, on_layer=None):
        """Run token rows (ids/pos/seq: int32 device tensors [n]) through all layers."""
        s = self.shape
        n = int(ids.shape[0])
        slot = (seq * cache.s_max + pos).to(torch.int32)
        st = self.new_state(n, pos, seq, slot, force_layer)
        if self.gpt2:
            B.embed_positions(n, s.d_model, s.vocab, s.max_pos, ids, pos, self.embed,
                              self.pos_embed, st.h[0])
        else:
            B.embed(n, s.d_model, s.vocab, ids, self.embed, st.h[0])
        B.token_init(n, s.n_layers, s.d_model, st.active[0], st.counts, st.exit_layer, st.inertia)
        args = self.layer_args(st, cache, cfg, attn_tiles)
        for i in range(1, s.n_layers + 1):
            B.layer_step(args, i)
            if on_layer is not None:
                on_layer(i, st)
        if logit_rows is None:
            return PassResult(None, None, st.exit_layer, st)
        rows = logit_rows.to(torch.int32)
        nr = int(rows.shape[0])
        n_rows = torch.tensor([nr], dtype=torch.int32, device=self.device)
        logits = torch.empty((nr, s.vocab), dtype=torch.float32, device=self.device)
        xn = torch.empty((nr, s.d_model), dtype=self.tdt, device=self.device)
        if self.gpt2:
            B.final_logits_layernorm(s.d_model, s.vocab, s.ln_eps, st.h[0], st.h[1],
                                     st.exit_layer, rows, n_rows, nr, self.final_ln_g,
                                     self.final_ln_b, self.lm_head, xn, logits)
        else:
            B.final_logits(s.d_model, s.vocab, s.rms_eps, st.h[0], st.h[1], st.exit_layer, rows,
                           n_rows, nr, self.final_norm, self.lm_head, xn, logits)
        return PassResult(logits, rows, st.exit_layer, st)

    def prefill(self, ids, cfg, s_max=None, force_layer=None, logits="all", cache=None,
                on_layer=None):
        """ids: [B, T] (numpy or tensor).  logits: "all", "last" or None."""
        ids = torch.as_tensor(np.asarray(ids) if not isinstance(ids, torch.Tensor) else ids)
        Bn, T = ids.shape
        s_max = T if s_max is None else s_max
        dev = self.device
        if cache is None:
            cache = self.new_cache(Bn, s_max)
        pos = torch.arange(T, dtype=torch.int32, device=dev).repeat(Bn)
        seq = torch.arange(Bn, dtype=torch.int32, device=dev).repeat_interleave(T)
        self._check_positions(pos, s_max, pos_max=T - 1)
        fl = None
        if isinstance(force_layer, torch.Tensor):
            fl = force_layer.reshape(-1).to(dev, torch.int32)
        elif force_layer is not None:
            fl = torch.as_tensor(np.asarray(force_layer).reshape(-1), dtype=torch.int32).to(dev)
        rows = None
        if logits == "all":
            rows = torch.arange(Bn * T, dtype=torch.int32, device=dev)
        elif logits == "last":
            rows = torch.arange(Bn, dtype=torch.int32, device=dev) * T + (T - 1)
        res = self.token_pass(ids.reshape(-1).to(dev, torch.int32), pos, seq, cache, cfg, fl,
                              True, rows, on_layer)
        return res, cache

    def decode_step(self, cache, ids, pos, cfg, force_layer=None, on_layer=None, pos_max=None):
        """One new token per sequence: ids, pos int32 device tensors [n_seq];
        pos_max: the largest position, when known on the host (no read-back)."""
        dev = self.device
        n = int(ids.shape[0])
        seq = torch.arange(n, dtype=torch.int32, device=dev)
        self._check_positions(pos, cache.s_max, pos_max)
        rows = torch.arange(n, dtype=torch.int32, device=dev)
        return self.token_pass(ids.to(torch.int32), pos.to(torch.int32), seq, cache, cfg,
                               force_layer, False, rows, on_layer)

    def greedy(self, logits):
        n, V = logits.shape
        out = torch.empty(n, dtype=torch.int32, device=self.device)
        B.argmax(n, V, logits, out)
        return out

    def generate(self, ids, n_steps, cfg, force_layer=None):
        """Prefill then n_steps greedy steps; returns (prefill result, [step results], ids [B, n_steps])."""
        ids_t = torch.as_tensor(np.asarray(ids))
        Bn, T = ids_t.shape
        res, cache = self.prefill(ids_t, cfg, s_max=T + n_steps, force_layer=force_layer,
                                  logits="last")
        nxt = self.greedy(res.logits)
        steps, out = [], []
        for k in range(n_steps):
            out.append(nxt)
            pos = torch.full((Bn,), T + k, dtype=torch.int32, device=self.device)
            st = self.decode_step(cache, nxt, pos, cfg, pos_max=T + k)
            steps.append(st)
            nxt = self.greedy(st.logits)
        gen = torch.stack(out, dim=1) if out else torch.zeros((Bn, 0), dtype=torch.int32)
        return res, steps, gen, cache


@dataclasses.dataclass
class ClassifyOutput:
    logits: torch.Tensor          # [B, n_classes] f32, from each [CLS] row at its exit
    exit_layer: torch.Tensor      # [B*T] int32 (n_layers: never exited)
    cls_exit_layer: torch.Tensor  # [B]
    state: dict                   # device buffers of the pass (h, inertia, sims, ...)


class EncoderModel:
    """A BERT-style post-norm encoder classifier held on the device (bf16),
    run with token-level exit in classification mode:

        adept_encoder_embed -> adept_token_init -> adept_encoder_layer_step(i),
        i = 1..N -> adept_classify_head

    weights: a dict like adept_inputs.encoder_weights() (numpy, per layer) or
    the same keys stacked over layers as torch tensors.
    """

    def __init__(self, shape, weights, device="cuda"):
        self.shape = shape
        self.device = torch.device(device)
        dev, tdt = self.device, torch.bfloat16

        def up(x):
            if isinstance(x, torch.Tensor):
                return x.to(dev, tdt).contiguous()
            return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev).to(tdt)

        L = weights["layers"]
        if isinstance(L, list):
            stack = lambda k: up(np.stack([lw[k] for lw in L]))
            self.w_qkv = up(np.stack([np.concatenate([lw["wq"], lw["wk"], lw["wv"]]) for lw in L]))
            self.b_qkv = up(np.stack([np.concatenate([lw["bq"], lw["bk"], lw["bv"]]) for lw in L]))
        else:
            stack = lambda k: up(L[k])
            self.w_qkv = up(torch.cat([L["wq"], L["wk"], L["wv"]], dim=1))
            self.b_qkv = up(torch.cat([L["bq"], L["bk"], L["bv"]], dim=1))
        self.w_o, self.b_o = stack("wo"), stack("bo")
        self.ln1_g, self.ln1_b = stack("ln1_g"), stack("ln1_b")
        self.w_in, self.b_in = stack("w_in"), stack("b_in")
        self.w_out, self.b_out = stack("w_out"), stack("b_out")
        self.ln2_g, self.ln2_b = stack("ln2_g"), stack("ln2_b")
        self.word = up(weights["word_embed"])
        self.pos_emb = up(weights["pos_embed"])
        self.type_emb = up(weights["type_embed"])
        self.eln_g, self.eln_b = up(weights["embed_ln_g"]), up(weights["embed_ln_b"])
        self.cls_w, self.cls_b = up(weights["cls_w"]), up(weights["cls_b"])

    def classify(self, ids, cfg, force_layer=None, state=None, on_layer=None, stop_at_cls=True):
        """ids [B, T] (numpy or tensor); cfg from binding.exit_cfg.  A state
        dict from an earlier call of the same shape is reused (no allocation).
        on_layer(i, state) is called after each layer step (read-back hook).
        stop_at_cls: a sequence's rows leave when its [CLS] row exits."""
        s, dev = self.shape, self.device
        ids = torch.as_tensor(np.asarray(ids) if not isinstance(ids, torch.Tensor) else ids)
        Bn, T = ids.shape
        n, D, Dq, F, N = Bn * T, s.d_model, s.d_q, s.d_ff, s.n_layers
        i32 = dict(dtype=torch.int32, device=dev)
        bf = dict(dtype=torch.bfloat16, device=dev)
        st = state
        if st is None or st["n"] != n:
            st = {
                "n": n,
                "h": [torch.empty((n, D), **bf) for _ in range(2)],
                "inertia": torch.empty((n, D), dtype=torch.float32, device=dev),
                "pos": torch.arange(T, **i32).repeat(Bn),
                "seq": torch.arange(Bn, **i32).repeat_interleave(T),
                "active": [torch.empty(n, **i32) for _ in range(2)],
                "counts": torch.zeros(4, **i32),
                "exited": torch.empty(n, **i32),
                "exit_layer": torch.empty(n, **i32),
                "exit_flag": torch.empty(max(n, 4), dtype=torch.uint8, device=dev),
                "sim_out": torch.empty(n, dtype=torch.float64, device=dev),
                "key_live": torch.empty(n, dtype=torch.uint8, device=dev),
                "key_len": torch.full((Bn,), T, **i32),
                "k_buf": torch.empty((n, Dq), **bf), "v_buf": torch.empty((n, Dq), **bf),
                "q_buf": torch.empty((n, Dq), **bf), "attn_out": torch.empty((n, Dq), **bf),
                "y_buf": torch.empty((n, D), **bf), "ffn_act": torch.empty((n, F), **bf),
                "logits": torch.empty((Bn, s.n_classes), dtype=torch.float32, device=dev),
                "workspace": None,
            }
        st["force"] = None
        if force_layer is not None:
            st["force"] = torch.as_tensor(np.asarray(force_layer).reshape(-1)
                                          if not isinstance(force_layer, torch.Tensor)
                                          else force_layer.reshape(-1)).to(dev, torch.int32)
        a = B.EncoderArgs()
        a.dtype, a.n_layers, a.d_model, a.n_heads = B.BF16, N, D, s.n_heads
        a.head_dim, a.d_ff, a.ln_eps, a.exit = s.head_dim, F, s.ln_eps, cfg
        for k in ("w_qkv", "b_qkv", "w_o", "b_o", "ln1_g", "ln1_b", "w_in", "b_in", "w_out",
                  "b_out", "ln2_g", "ln2_b"):
            setattr(a, k, B.ptr(getattr(self, k)))
        a.n_tok, a.n_seq, a.seq_len = n, Bn, T
        a.cls_stop = int(bool(stop_at_cls))
        a.h[0], a.h[1] = B.ptr(st["h"][0]), B.ptr(st["h"][1])
        a.inertia, a.pos, a.seq = B.ptr(st["inertia"]), B.ptr(st["pos"]), B.ptr(st["seq"])
        a.active[0], a.active[1] = B.ptr(st["active"][0]), B.ptr(st["active"][1])
        cp = B.ptr(st["counts"])
        a.n_active[0], a.n_active[1], a.n_exited = cp, cp + 4, cp + 8
        a.exited, a.exit_layer = B.ptr(st["exited"]), B.ptr(st["exit_layer"])
        a.exit_flag, a.sim_out = B.ptr(st["exit_flag"]), B.ptr(st["sim_out"])
        a.force_layer = B.ptr(st["force"])
        a.key_live, a.key_len = B.ptr(st["key_live"]), B.ptr(st["key_len"])
        for k in ("k_buf", "v_buf", "q_buf", "attn_out", "y_buf", "ffn_act"):
            setattr(a, k, B.ptr(st[k]))
        need = B.encoder_workspace_bytes(a)
        if st["workspace"] is None or st["workspace"].numel() < need:
            st["workspace"] = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
        a.workspace, a.workspace_bytes = B.ptr(st["workspace"]), st["workspace"].numel()

        ids_d = ids.reshape(-1).to(dev, torch.int32)
        B.encoder_embed(n, D, s.vocab, s.max_pos, s.ln_eps, ids_d, st["pos"], self.word,
                        self.pos_emb, self.type_emb, self.eln_g, self.eln_b, st["h"][0])
        B.token_init(n, N, D, st["active"][0], st["counts"], st["exit_layer"], st["inertia"])
        st["key_live"].fill_(1)
        for i in range(1, N + 1):
            B.encoder_layer_step(a, i)
            if on_layer is not None:
                on_layer(i, st)
        B.classify_head(Bn, T, D, s.n_classes, st["h"][0], st["h"][1], st["exit_layer"],
                        self.cls_w, self.cls_b, st["logits"])
        return ClassifyOutput(st["logits"], st["exit_layer"], st["exit_layer"][::T], st)
