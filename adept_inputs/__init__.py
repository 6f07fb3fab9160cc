"""Seeded synthetic inputs shared by the oracle, the tests and the bench.

This module holds data only: shapes of the workloads and seeded random
draws.  It contains none of the method's arithmetic (no norm, projection,
attention, similarity or compaction), so that the CPU oracle and the HIP
path can both consume its arrays without sharing any computation.

Every generator is deterministic in (seed, tensor name): each tensor gets
its own numpy PCG64 stream derived from the master seed and a CRC of the
name, so adding a tensor never shifts the values of another.

Values meant for a bf16 run are produced as float32 arrays whose entries are
exactly representable in bfloat16 (round-to-nearest-even of the float32
draw, done by torch's dtype conversion), so both sides see identical numbers.
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np

__all__ = [
    "DecoderShape", "EncoderShape", "TINY", "LLAMA7B", "BERT_BASE", "GPT2_XL",
    "rng", "to_bf16_values", "decoder_weights", "gpt2_weights", "encoder_weights",
    "decoder_weights_torch", "gpt2_weights_torch",
    "token_ids", "normal", "gains",
]


@dataclasses.dataclass(frozen=True)
class DecoderShape:
    """Pre-norm decoder.  family "llama": RMSNorm, rotary positions, SwiGLU,
    no biases, untied LM head.  family "gpt2": LayerNorm with bias (eps
    ln_eps), learned absolute positions (max_pos), tanh-approximated GELU
    MLP, biases on every projection, LM head tied to the token embedding."""
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    family: str = "llama"
    max_pos: int = 0
    ln_eps: float = 1e-5

    @property
    def d_q(self) -> int:
        return self.n_heads * self.head_dim


@dataclasses.dataclass(frozen=True)
class EncoderShape:
    """BERT-style post-norm encoder (LayerNorm, learned positions, GELU)."""
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    max_pos: int
    n_classes: int = 2
    ln_eps: float = 1e-12

    @property
    def d_q(self) -> int:
        return self.n_heads * self.head_dim


# The workload shapes: a tiny decoder that the oracle runs in seconds, the
# 7B-class decoder (32 layers, width 4096, 32 heads of 128, FFN 11008,
# vocab 32000) and a BERT-base-class encoder (12 layers, width 768).
TINY = DecoderShape(n_layers=4, d_model=256, n_heads=4, head_dim=64, d_ff=1024, vocab=1024)
# GPT2-XL-shaped decoder: 48 layers, width 1600 = 25 heads of 64, MLP 6400,
# 1024 positions; the vocabulary is padded from 50257 to 50304 (a multiple of
# 64) as GPT-2 training code commonly does
GPT2_XL = DecoderShape(n_layers=48, d_model=1600, n_heads=25, head_dim=64, d_ff=6400,
                       vocab=50304, family="gpt2", max_pos=1024)
LLAMA7B = DecoderShape(n_layers=32, d_model=4096, n_heads=32, head_dim=128, d_ff=11008, vocab=32000)
BERT_BASE = EncoderShape(n_layers=12, d_model=768, n_heads=12, head_dim=64, d_ff=3072,
                         vocab=30522, max_pos=512)


def rng(seed: int, name: str) -> np.random.Generator:
    """Independent PCG64 stream for tensor `name` under master `seed`."""
    return np.random.Generator(np.random.PCG64([seed & 0xFFFFFFFF, zlib.crc32(name.encode())]))


def to_bf16_values(x: np.ndarray) -> np.ndarray:
    """float32 array of the bfloat16 values nearest to x (RNE, via torch)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _finish(x: np.ndarray, dtype: str) -> np.ndarray:
    x = x.astype(np.float32)
    if dtype == "bf16":
        return to_bf16_values(x)
    if dtype != "f32":
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    return x


def normal(seed: int, name: str, shape, std: float = 1.0, mean: float = 0.0,
           dtype: str = "f32") -> np.ndarray:
    """N(mean, std^2) draws of `shape`."""
    x = rng(seed, name).standard_normal(size=shape, dtype=np.float32)
    return _finish(x * np.float32(std) + np.float32(mean), dtype)


def gains(seed: int, name: str, shape, dtype: str = "f32") -> np.ndarray:
    """Norm gains 1 + 0.1 N(0,1): non-unit so that a gain applied to the
    wrong channel or layer changes the result."""
    return normal(seed, name, shape, std=0.1, mean=1.0, dtype=dtype)


def token_ids(seed: int, vocab: int, batch: int, length: int, name: str = "ids") -> np.ndarray:
    """Uniform token ids in [0, vocab), shape [batch, length], int32."""
    return rng(seed, name).integers(0, vocab, size=(batch, length), dtype=np.int64).astype(np.int32)


def decoder_weights(shape: DecoderShape, seed: int, dtype: str = "f32", std: float = 0.02) -> dict:
    """Random-init weights of a Llama-style decoder.

    Linear weights and the embedding are N(0, std^2) in nn.Linear
    [out_features, in_features] order; norm gains are 1 + 0.1 N(0,1).
    Returns {"embed", "final_norm", "lm_head", "layers": [per-layer dict]}
    with per-layer keys attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up,
    w_down.
    """
    D, Dq, F, V = shape.d_model, shape.d_q, shape.d_ff, shape.vocab
    out = {
        "embed": normal(seed, "embed", (V, D), std, dtype=dtype),
        "final_norm": gains(seed, "final_norm", (D,), dtype),
        "lm_head": normal(seed, "lm_head", (V, D), std, dtype=dtype),
        "layers": [],
    }
    for i in range(1, shape.n_layers + 1):
        p = f"layer{i}."
        out["layers"].append({
            "attn_norm": gains(seed, p + "attn_norm", (D,), dtype),
            "wq": normal(seed, p + "wq", (Dq, D), std, dtype=dtype),
            "wk": normal(seed, p + "wk", (Dq, D), std, dtype=dtype),
            "wv": normal(seed, p + "wv", (Dq, D), std, dtype=dtype),
            "wo": normal(seed, p + "wo", (D, Dq), std, dtype=dtype),
            "ffn_norm": gains(seed, p + "ffn_norm", (D,), dtype),
            "w_gate": normal(seed, p + "w_gate", (F, D), std, dtype=dtype),
            "w_up": normal(seed, p + "w_up", (F, D), std, dtype=dtype),
            "w_down": normal(seed, p + "w_down", (D, F), std, dtype=dtype),
        })
    return out


def gpt2_weights(shape: DecoderShape, seed: int, dtype: str = "f32", std: float = 0.02) -> dict:
    """Random-init weights of a GPT-2-style decoder (family "gpt2").

    Linear weights, biases and the token / position embeddings N(0, std^2)
    in nn.Linear [out_features, in_features] order (biases and LayerNorm
    shifts non-zero on purpose, so that a dropped one is visible); LayerNorm
    gains 1 + 0.1 N(0,1).  The LM head is the token embedding (tied).
    Returns {"embed", "pos_embed", "final_ln_g", "final_ln_b", "layers"} with
    per-layer keys ln1_g, ln1_b, wq, wk, wv, bq, bk, bv, wo, bo, ln2_g, ln2_b,
    w_fc, b_fc, w_proj, b_proj.
    """
    D, Dq, F, V = shape.d_model, shape.d_q, shape.d_ff, shape.vocab
    out = {
        "embed": normal(seed, "wte", (V, D), std, dtype=dtype),
        "pos_embed": normal(seed, "wpe", (shape.max_pos, D), std, dtype=dtype),
        "final_ln_g": gains(seed, "ln_f.g", (D,), dtype),
        "final_ln_b": normal(seed, "ln_f.b", (D,), std, dtype=dtype),
        "layers": [],
    }
    for i in range(1, shape.n_layers + 1):
        p = f"h{i}."
        lay = {}
        for nm, shp in (("wq", (Dq, D)), ("wk", (Dq, D)), ("wv", (Dq, D)), ("wo", (D, Dq)),
                        ("w_fc", (F, D)), ("w_proj", (D, F))):
            lay[nm] = normal(seed, p + nm, shp, std, dtype=dtype)
        for nm, n in (("bq", Dq), ("bk", Dq), ("bv", Dq), ("bo", D), ("b_fc", F), ("b_proj", D),
                      ("ln1_b", D), ("ln2_b", D)):
            lay[nm] = normal(seed, p + nm, (n,), std, dtype=dtype)
        lay["ln1_g"] = gains(seed, p + "ln1_g", (D,), dtype)
        lay["ln2_g"] = gains(seed, p + "ln2_g", (D,), dtype)
        out["layers"].append(lay)
    return out


def encoder_weights(shape: EncoderShape, seed: int, dtype: str = "f32", std: float = 0.02) -> dict:
    """Random-init weights of a BERT-style post-norm encoder with a linear
    classification head on the first ([CLS]) position.

    Linear weights, biases and embeddings are N(0, std^2) (biases non-zero
    on purpose, so that a dropped bias is visible); LayerNorm gains are
    1 + 0.1 N(0,1) and shifts N(0, std^2).
    """
    D, Dq, F, V = shape.d_model, shape.d_q, shape.d_ff, shape.vocab
    out = {
        "word_embed": normal(seed, "word_embed", (V, D), std, dtype=dtype),
        "pos_embed": normal(seed, "pos_embed", (shape.max_pos, D), std, dtype=dtype),
        "type_embed": normal(seed, "type_embed", (D,), std, dtype=dtype),
        "embed_ln_g": gains(seed, "embed_ln_g", (D,), dtype),
        "embed_ln_b": normal(seed, "embed_ln_b", (D,), std, dtype=dtype),
        "cls_w": normal(seed, "cls_w", (shape.n_classes, D), std, dtype=dtype),
        "cls_b": normal(seed, "cls_b", (shape.n_classes,), std, dtype=dtype),
        "layers": [],
    }
    for i in range(1, shape.n_layers + 1):
        p = f"layer{i}."
        lay = {}
        for nm, shp in (("wq", (Dq, D)), ("wk", (Dq, D)), ("wv", (Dq, D)), ("wo", (D, Dq)),
                        ("w_in", (F, D)), ("w_out", (D, F))):
            lay[nm] = normal(seed, p + nm, shp, std, dtype=dtype)
        for nm, n in (("bq", Dq), ("bk", Dq), ("bv", Dq), ("bo", D), ("b_in", F), ("b_out", D),
                      ("ln1_b", D), ("ln2_b", D)):
            lay[nm] = normal(seed, p + nm, (n,), std, dtype=dtype)
        lay["ln1_g"] = gains(seed, p + "ln1_g", (D,), dtype)
        lay["ln2_g"] = gains(seed, p + "ln2_g", (D,), dtype)
        out["layers"].append(lay)
    return out


def _torch_fillers(seed, device, dtype, n_layers):
    """(single, stacked): N(mean, scale^2) tensors on `device` from torch's
    counter-based generator, seeded per name (and per layer for stacked
    [n_layers, ...] tensors, "layer{i}.{name}"), so any slice can be
    regenerated alone."""
    import torch
    g = torch.Generator(device=device)

    def fill(out, name, scale, mean):
        g.manual_seed((seed * 1000003 + zlib.crc32(name.encode())) & 0x7FFFFFFFFFFFFFFF)
        tmp = torch.randn(out.shape, generator=g, device=device, dtype=torch.float32)
        out.copy_(tmp.mul_(scale).add_(mean))

    def stacked(name, shp, scale, mean=0.0):
        out = torch.empty((n_layers,) + shp, dtype=dtype, device=device)
        for i in range(n_layers):
            fill(out[i], f"layer{i + 1}.{name}", scale, mean)
        return out

    def single(name, shp, scale, mean=0.0):
        out = torch.empty(shp, dtype=dtype, device=device)
        fill(out, name, scale, mean)
        return out

    return single, stacked


def decoder_weights_torch(shape: DecoderShape, seed: int, device, dtype=None, std: float = 0.02):
    """Random-init decoder weights generated directly on `device` (torch's
    counter-based generator), stacked over layers: attn_norm/ffn_norm [N, D],
    wq/wk/wv [N, Dq, D], wo [N, D, Dq], w_gate/w_up [N, F, D], w_down [N, D, F],
    embed/lm_head [V, D], final_norm [D].  Linear weights N(0, std^2), gains
    1 + 0.1 N(0,1).  Each layer slice has its own seed, so any layer can be
    regenerated alone.  Used for the 7B-class shapes, whose weights are too
    large to draw on the host.
    """
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    N, D, Dq, F, V = shape.n_layers, shape.d_model, shape.d_q, shape.d_ff, shape.vocab
    single, stacked = _torch_fillers(seed, device, dtype, N)
    return {
        "embed": single("embed", (V, D), std),
        "final_norm": single("final_norm", (D,), 0.1, 1.0),
        "lm_head": single("lm_head", (V, D), std),
        "attn_norm": stacked("attn_norm", (D,), 0.1, 1.0),
        "wq": stacked("wq", (Dq, D), std),
        "wk": stacked("wk", (Dq, D), std),
        "wv": stacked("wv", (Dq, D), std),
        "wo": stacked("wo", (D, Dq), std),
        "ffn_norm": stacked("ffn_norm", (D,), 0.1, 1.0),
        "w_gate": stacked("w_gate", (F, D), std),
        "w_up": stacked("w_up", (F, D), std),
        "w_down": stacked("w_down", (D, F), std),
    }


def gpt2_weights_torch(shape: DecoderShape, seed: int, device, dtype=None, std: float = 0.02):
    """gpt2_weights() drawn directly on `device` (torch's generator, as
    decoder_weights_torch), stacked over layers: ln1_g/ln1_b/ln2_g/ln2_b,
    bo/b_proj [N, D], wq/wk/wv [N, Dq, D], bq/bk/bv [N, Dq], wo [N, D, Dq],
    w_fc [N, F, D], b_fc [N, F], w_proj [N, D, F]; embed [V, D] (also the
    head), pos_embed [max_pos, D], final_ln_g/final_ln_b [D].  For the
    GPT2-XL shape, whose 1.5 G weights are slow to draw on the host."""
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    N, D, Dq, F, V = shape.n_layers, shape.d_model, shape.d_q, shape.d_ff, shape.vocab
    single, stacked = _torch_fillers(seed, device, dtype, N)
    out = {
        "embed": single("wte", (V, D), std),
        "pos_embed": single("wpe", (shape.max_pos, D), std),
        "final_ln_g": single("ln_f.g", (D,), 0.1, 1.0),
        "final_ln_b": single("ln_f.b", (D,), std),
    }
    for nm, shp in (("wq", (Dq, D)), ("wk", (Dq, D)), ("wv", (Dq, D)), ("wo", (D, Dq)),
                    ("w_fc", (F, D)), ("w_proj", (D, F)), ("bq", (Dq,)), ("bk", (Dq,)),
                    ("bv", (Dq,)), ("bo", (D,)), ("b_fc", (F,)), ("b_proj", (D,)),
                    ("ln1_b", (D,)), ("ln2_b", (D,))):
        out[nm] = stacked(nm, shp, std)
    out["ln1_g"] = stacked("ln1_g", (D,), 0.1, 1.0)
    out["ln2_g"] = stacked("ln2_g", (D,), 0.1, 1.0)
    return out


def hsm_weights(d_model: int, seed: int, dtype: str = "f32", std: float = 0.02) -> dict:
    """Random-init weights of a hidden state mapper of width D (the layer list
    of Table S1): fully connected weights N(0, std^2) in [out, in] order,
    biases N(0, std^2), the three norm gains 1 + 0.1 N(0,1), a 3 x 3
    convolution kernel N(0, 0.25) and its scalar bias N(0, 0.01) (f32)."""
    D = d_model
    return {
        "g0": gains(seed, "hsm.g0", (D,), dtype),
        "conv": normal(seed, "hsm.conv", (3, 3), 0.5, dtype="f32"),
        "conv_b": float(normal(seed, "hsm.conv_b", (1,), 0.1, dtype="f32")[0]),
        "w1": normal(seed, "hsm.w1", (4 * D, D), std, dtype=dtype),
        "b1": normal(seed, "hsm.b1", (4 * D,), std, dtype=dtype),
        "w2": normal(seed, "hsm.w2", (8 * D, 4 * D), std, dtype=dtype),
        "b2": normal(seed, "hsm.b2", (8 * D,), std, dtype=dtype),
        "w3": normal(seed, "hsm.w3", (4 * D, 8 * D), std, dtype=dtype),
        "b3": normal(seed, "hsm.b3", (4 * D,), std, dtype=dtype),
        "g1": gains(seed, "hsm.g1", (4 * D,), dtype),
        "w4": normal(seed, "hsm.w4", (D, 4 * D), std, dtype=dtype),
        "b4": normal(seed, "hsm.b4", (D,), std, dtype=dtype),
        "g2": gains(seed, "hsm.g2", (D,), dtype),
    }


def forced_exit_layers(seed: int, n: int, lo: int, hi: int) -> np.ndarray:
    """Seeded exit schedule: exit layer of each of n tokens uniform in [lo, hi]."""
    return rng(seed, "forced_exit").integers(lo, hi + 1, size=n).astype(np.int32)
