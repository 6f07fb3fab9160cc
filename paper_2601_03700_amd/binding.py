"""ctypes binding of libadept.so (the C ABI in include/adept.h).

Argument marshalling only: every function takes torch tensors (device
memory) or None, passes their data pointers and the current HIP stream to the
library, and raises AdeptError on a non-zero status.  No computation happens
here.  Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libadept.so")

F32, BF16 = 0, 1
FAMILY_LLAMA, FAMILY_GPT2 = 0, 1
SIM_GLOBAL, SIM_LOCAL, SIM_BOTH = 0, 1, 2
METRICS = {"global": SIM_GLOBAL, "local": SIM_LOCAL, "both": SIM_BOTH}

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t


class AdeptError(RuntimeError):
    pass


class ExitCfg(ctypes.Structure):
    _fields_ = [("delta", ctypes.c_double), ("min_exit_layer", _i32), ("n_layers", _i32),
                ("metric", _i32), ("prompt_level", _i32)]


class HsmWeights(ctypes.Structure):
    _fields_ = [("g0", _vp), ("conv", (ctypes.c_float * 3) * 3), ("conv_bias", ctypes.c_float),
                ("w1", _vp), ("b1", _vp), ("w2", _vp), ("b2", _vp), ("w3", _vp), ("b3", _vp),
                ("g1", _vp), ("w4", _vp), ("b4", _vp), ("g2", _vp)]


class LayerArgs(ctypes.Structure):
    _fields_ = [
        ("dtype", _i32), ("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32),
        ("head_dim", _i32), ("d_ff", _i32), ("rms_eps", ctypes.c_float), ("exit", ExitCfg),
        ("w_qkv", _vp), ("w_o", _vp), ("w_gate", _vp),
        ("w_up", _vp), ("w_down", _vp), ("rope_cos", _vp), ("rope_sin", _vp),
        ("rope_max_pos", _i32),
        ("n_tok", _i32), ("max_active", _i32), ("n_seq", _i32), ("s_max", _i32),
        ("attn_tiles", _i32),
        ("h", _vp * 2), ("inertia", _vp), ("pos", _vp), ("seq", _vp), ("slot", _vp),
        ("active", _vp * 2), ("n_active", _vp * 2), ("exited", _vp), ("n_exited", _vp),
        ("exit_layer", _vp), ("exit_flag", _vp), ("sim_out", _vp), ("force_layer", _vp),
        ("k_cache", _vp), ("v_cache", _vp), ("n_slots", _i64),
        ("q_buf", _vp), ("attn_out", _vp), ("ffn_act", _vp),
        ("workspace", _vp), ("workspace_bytes", _sz), ("hsm", _vp),
        ("family", _i32), ("b_qkv", _vp), ("b_o", _vp), ("b_fc", _vp), ("b_proj", _vp),
        ("kv_fused", _i32),
    ]


class EncoderArgs(ctypes.Structure):
    _fields_ = [
        ("dtype", _i32), ("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32),
        ("head_dim", _i32), ("d_ff", _i32), ("ln_eps", ctypes.c_float), ("exit", ExitCfg),
        ("w_qkv", _vp), ("b_qkv", _vp), ("w_o", _vp), ("b_o", _vp), ("ln1_g", _vp),
        ("ln1_b", _vp), ("w_in", _vp), ("b_in", _vp), ("w_out", _vp), ("b_out", _vp),
        ("ln2_g", _vp), ("ln2_b", _vp),
        ("n_tok", _i32), ("n_seq", _i32), ("seq_len", _i32), ("cls_stop", _i32),
        ("h", _vp * 2), ("inertia", _vp), ("pos", _vp), ("seq", _vp),
        ("active", _vp * 2), ("n_active", _vp * 2), ("exited", _vp), ("n_exited", _vp),
        ("exit_layer", _vp), ("exit_flag", _vp), ("sim_out", _vp), ("force_layer", _vp),
        ("key_live", _vp), ("key_len", _vp), ("k_buf", _vp), ("v_buf", _vp), ("q_buf", _vp),
        ("attn_out", _vp), ("y_buf", _vp), ("ffn_act", _vp),
        ("workspace", _vp), ("workspace_bytes", _sz),
    ]


_SIGS = {
    "adept_abi_version": (_i32, []),
    "adept_last_error": (ctypes.c_char_p, []),
    "adept_rope_table": (_i32, [_i32, _i32, ctypes.c_double, _vp, _vp, _vp]),
    "adept_exit_test": (_i32, [_i32, _i32, _i32, ctypes.POINTER(ExitCfg), _vp, _vp, _i32, _vp,
                               _vp, _vp, _vp, _vp, _vp, _vp]),
    "adept_compact_workspace_bytes": (_sz, [_i32]),
    "adept_hsm_workspace_bytes": (_sz, [_i32, _i32]),
    "adept_hsm_forward": (_i32, [_i32, _i32, ctypes.c_float, ctypes.POINTER(HsmWeights), _vp, _vp,
                                 _i32, _vp, _vp, _vp, _i32, _vp, _vp, _sz, _vp]),
    "adept_exit_prompt_level_workspace_bytes": (_sz, [_i32]),
    "adept_exit_prompt_level": (_i32, [_vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _sz, _vp]),
    "adept_compact": (_i32, [_i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _sz,
                             _vp]),
    "adept_kv_generate_workspace_bytes": (_sz, [_i32, _i32]),
    "adept_kv_generate": (_i32, [_i32, _i32, _i32, _i32, _i32, ctypes.c_float, _vp, _vp, _vp,
                                 _i32, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _i32, _vp, _vp,
                                 _i64, _vp, _sz, _vp]),
    "adept_kv_generate_noalloc": (_i32, [_i32, _i32, _i32, _i32, _i32, ctypes.c_float, _vp, _vp,
                                         _vp, _i32, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _i32,
                                         _vp, _vp, _i64, _vp]),
    "adept_kv_generate_layernorm_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "adept_kv_generate_layernorm": (_i32, [_i32, _i32, _i32, _i32, _i32, ctypes.c_float, _vp, _vp,
                                           _vp, _i32, _vp, _vp, _vp, _i64, _vp, _i64, _vp, _vp,
                                           _i64, _vp, _sz, _vp]),
    "adept_fold_bias": (_i32, [_i32, _i32, _i32, _i32, _vp, _i64, _vp, _i64, _vp, _i64, _vp]),
    "adept_embed_positions": (_i32, [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "adept_final_logits_layernorm": (_i32, [_i32, _i32, _i32, ctypes.c_float, _vp, _vp, _vp, _vp,
                                            _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "adept_attend_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "adept_attend": (_i32, [_i32, _i32, _i32, ctypes.c_float, _i32, _vp, _vp, _vp, _i32, _vp,
                            _vp, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "adept_layer_workspace_bytes": (_sz, [ctypes.POINTER(LayerArgs)]),
    "adept_layer_step": (_i32, [ctypes.POINTER(LayerArgs), _i32, _vp]),
    "adept_embed": (_i32, [_i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "adept_final_logits": (_i32, [_i32, _i32, _i32, ctypes.c_float, _vp, _vp, _vp, _vp, _vp,
                                  _i32, _vp, _vp, _vp, _vp, _vp]),
    "adept_argmax": (_i32, [_i32, _i32, _vp, _vp, _vp]),
    "adept_token_init": (_i32, [_i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "adept_fold_gain": (_i32, [_i32, _i32, _i32, _i32, _vp, _i64, _vp, _i64, _vp]),
    "adept_encoder_workspace_bytes": (_sz, [ctypes.POINTER(EncoderArgs)]),
    "adept_encoder_layer_step": (_i32, [ctypes.POINTER(EncoderArgs), _i32, _vp]),
    "adept_encoder_embed": (_i32, [_i32, _i32, _i32, _i32, ctypes.c_float, _vp, _vp, _vp, _vp,
                                   _vp, _vp, _vp, _vp, _vp]),
    "adept_classify_head": (_i32, [_i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "adept_timing_enable": (_i32, [_i32]),
    "adept_timing_select": (_i32, [ctypes.c_char_p]),
    "adept_timing_reset": (None, []),
    "adept_timing_count": (_i32, []),
    "adept_timing_get": (_i32, [_i32, ctypes.c_char_p, _i32, ctypes.POINTER(_i64),
                                ctypes.POINTER(ctypes.c_double)]),
}

EXPORTED = tuple(_SIGS)
_lib = None


def lib():
    """Load libadept.so once (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise AdeptError(f"{LIB_PATH} not built: run python -m paper_2601_03700_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status, what):
    if status != 0:
        msg = lib().adept_last_error().decode(errors="replace")
        raise AdeptError(f"{what} failed with status {status}: {msg}")


def ptr(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def stream_handle(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def dtype_code(t_or_str):
    if isinstance(t_or_str, str):
        return {"f32": F32, "bf16": BF16}[t_or_str]
    return {torch.float32: F32, torch.bfloat16: BF16}[t_or_str.dtype]


def exit_cfg(delta, n_layers, metric="global", min_exit_layer=1, prompt_level=False):
    return ExitCfg(float(delta), int(min_exit_layer), int(n_layers), METRICS[metric],
                   int(bool(prompt_level)))


# ----------------------------------------------------------------------------
# thin wrappers, one per entry point
# ----------------------------------------------------------------------------

def rope_table(max_pos, head_dim, theta, cos_out, sin_out, stream=None):
    _check(lib().adept_rope_table(max_pos, head_dim, theta, ptr(cos_out), ptr(sin_out),
                                  stream_handle(stream)), "adept_rope_table")


def exit_test(d_model, layer, cfg, active_rows, n_active, max_active, h_cur, h_prev, inertia,
              force_layer, exit_flag, sim_out=None, stream=None):
    _check(lib().adept_exit_test(dtype_code(h_cur), d_model, layer, ctypes.byref(cfg),
                                 ptr(active_rows), ptr(n_active), max_active, ptr(h_cur),
                                 ptr(h_prev), ptr(inertia), ptr(force_layer), ptr(exit_flag),
                                 ptr(sim_out), stream_handle(stream)), "adept_exit_test")


def exit_prompt_level_workspace_bytes(n_seq):
    return lib().adept_exit_prompt_level_workspace_bytes(n_seq)


def exit_prompt_level(active_rows, n_active, max_active, seq, pos, n_seq, exit_flag,
                      workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().adept_exit_prompt_level(ptr(active_rows), ptr(n_active), max_active, ptr(seq),
                                         ptr(pos), n_seq, ptr(exit_flag), ptr(workspace),
                                         ws_bytes, stream_handle(stream)),
           "adept_exit_prompt_level")


def hsm_weights(w):
    """HsmWeights from a dict of device tensors (bf16 matrices, biases and
    gains) plus the host 3x3 "conv" values and the "conv_b" scalar.  Keep the
    dict alive while the struct is used."""
    hw = HsmWeights()
    for k in ("g0", "w1", "b1", "w2", "b2", "w3", "b3", "g1", "w4", "b4", "g2"):
        setattr(hw, k, ptr(w[k]))
    for r in range(3):
        for t in range(3):
            hw.conv[r][t] = float(w["conv"][r][t])
    hw.conv_bias = float(w["conv_b"])
    return hw


def hsm_workspace_bytes(d_model, max_rows):
    return lib().adept_hsm_workspace_bytes(d_model, max_rows)


def hsm_forward(d_model, eps, hw, rows, n_rows, max_rows, h_cur, h_prev, inertia,
                inertia_updated, out, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().adept_hsm_forward(dtype_code(h_cur), d_model, eps, ctypes.byref(hw), ptr(rows),
                                   ptr(n_rows), max_rows, ptr(h_cur), ptr(h_prev), ptr(inertia),
                                   int(inertia_updated), ptr(out), ptr(workspace), ws_bytes,
                                   stream_handle(stream)),
           "adept_hsm_forward")


def compact_workspace_bytes(max_active):
    return lib().adept_compact_workspace_bytes(max_active)


def compact(layer, n_layers, exit_flag, active_rows, n_active, max_active, next_rows, n_next,
            exited_rows, n_exited, exit_layer, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().adept_compact(layer, n_layers, ptr(exit_flag), ptr(active_rows), ptr(n_active), max_active,
                               ptr(next_rows), ptr(n_next), ptr(exited_rows), ptr(n_exited),
                               ptr(exit_layer), ptr(workspace), ws_bytes, stream_handle(stream)),
           "adept_compact")


def kv_generate_workspace_bytes(n_layers, max_rows):
    return lib().adept_kv_generate_workspace_bytes(n_layers, max_rows)


def kv_generate(n_layers, d_model, n_heads, head_dim, eps, s_map, rows, n_rows, max_rows,
                exit_layer, cache_slot, pos, w_kv, w_kv_layer_stride, attn_gain, rope_cos,
                rope_sin, k_cache, v_cache, n_slots, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().adept_kv_generate(dtype_code(s_map), n_layers, d_model, n_heads, head_dim, eps,
                                   ptr(s_map), ptr(rows), ptr(n_rows), max_rows, ptr(exit_layer),
                                   ptr(cache_slot), ptr(pos), ptr(w_kv), w_kv_layer_stride,
                                   ptr(attn_gain), ptr(rope_cos), ptr(rope_sin),
                                   rope_cos.shape[0], ptr(k_cache), ptr(v_cache), n_slots,
                                   ptr(workspace), ws_bytes, stream_handle(stream)),
           "adept_kv_generate")


def kv_generate_noalloc(n_layers, d_model, n_heads, head_dim, eps, s_map, rows, n_rows, max_rows,
                        exit_layer, cache_slot, pos, w_kv, w_kv_layer_stride, attn_gain,
                        rope_cos, rope_sin, k_cache, v_cache, n_slots, stream=None):
    _check(lib().adept_kv_generate_noalloc(dtype_code(s_map), n_layers, d_model, n_heads,
                                           head_dim, eps, ptr(s_map), ptr(rows), ptr(n_rows),
                                           max_rows, ptr(exit_layer), ptr(cache_slot), ptr(pos),
                                           ptr(w_kv), w_kv_layer_stride, ptr(attn_gain),
                                           ptr(rope_cos), ptr(rope_sin), rope_cos.shape[0],
                                           ptr(k_cache), ptr(v_cache), n_slots,
                                           stream_handle(stream)),
           "adept_kv_generate_noalloc")


def kv_generate_layernorm_workspace_bytes(n_layers, max_rows, d_model):
    return lib().adept_kv_generate_layernorm_workspace_bytes(n_layers, max_rows, d_model)


def kv_generate_layernorm(n_layers, d_model, n_heads, head_dim, eps, s_map, rows, n_rows,
                          max_rows, exit_layer, cache_slot, w_kv, w_kv_layer_stride, b_kv,
                          b_kv_layer_stride, k_cache, v_cache, n_slots, workspace=None,
                          stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().adept_kv_generate_layernorm(dtype_code(s_map), n_layers, d_model, n_heads,
                                             head_dim, eps, ptr(s_map), ptr(rows), ptr(n_rows),
                                             max_rows, ptr(exit_layer), ptr(cache_slot),
                                             ptr(w_kv), w_kv_layer_stride, ptr(b_kv),
                                             b_kv_layer_stride, ptr(k_cache), ptr(v_cache),
                                             n_slots, ptr(workspace), ws_bytes,
                                             stream_handle(stream)),
           "adept_kv_generate_layernorm")


def fold_bias(w, shift, bias, stream=None):
    """In place: bias[l][o] += sum_c w[l][o][c] * shift[l][c] for a stacked
    w [L, rows, cols] (rows contiguous), shift [L, cols] and bias [L, rows]
    (row views with unit column stride)."""
    L, rows, cols = w.shape
    assert w.stride(2) == 1 and (rows == 1 or w.stride(1) == cols)
    assert shift.stride(-1) == 1 and bias.stride(-1) == 1 and bias.shape[-1] == rows
    _check(lib().adept_fold_bias(dtype_code(w), L, rows, cols, ptr(w), w.stride(0), ptr(shift),
                                 shift.stride(0), ptr(bias), bias.stride(0),
                                 stream_handle(stream)), "adept_fold_bias")


def embed_positions(n, d_model, vocab, max_pos, ids, pos, wte, wpe, h0, stream=None):
    _check(lib().adept_embed_positions(dtype_code(wte), n, d_model, vocab, max_pos, ptr(ids),
                                       ptr(pos), ptr(wte), ptr(wpe), ptr(h0),
                                       stream_handle(stream)), "adept_embed_positions")


def final_logits_layernorm(d_model, vocab, eps, h0, h1, exit_layer, rows, n_rows, max_rows, ln_g,
                           ln_b, lm_head, x_norm, logits, stream=None):
    _check(lib().adept_final_logits_layernorm(dtype_code(h0), d_model, vocab, eps, ptr(h0),
                                              ptr(h1), ptr(exit_layer), ptr(rows), ptr(n_rows),
                                              max_rows, ptr(ln_g), ptr(ln_b), ptr(lm_head),
                                              ptr(x_norm), ptr(logits), stream_handle(stream)),
           "adept_final_logits_layernorm")


def attend_workspace_bytes(max_active, n_seq, n_heads, head_dim, s_max):
    return lib().adept_attend_workspace_bytes(max_active, n_seq, n_heads, head_dim, s_max)


def attend(n_heads, head_dim, q, rows, n_active, max_active, pos, seq, n_seq, k_layer, v_layer,
           s_max, out, causal=True, key_len=None, key_live=None, workspace=None, scale=None,
           stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    scale = 1.0 / math.sqrt(head_dim) if scale is None else scale
    _check(lib().adept_attend(dtype_code(q), n_heads, head_dim, scale, int(bool(causal)), ptr(q),
                              ptr(rows), ptr(n_active), max_active, ptr(pos), ptr(seq), n_seq,
                              ptr(k_layer), ptr(v_layer), s_max, ptr(key_len), ptr(key_live),
                              ptr(out), ptr(workspace), ws_bytes, stream_handle(stream)),
           "adept_attend")


def layer_workspace_bytes(args: LayerArgs):
    return lib().adept_layer_workspace_bytes(ctypes.byref(args))


def layer_step(args: LayerArgs, layer, stream=None):
    _check(lib().adept_layer_step(ctypes.byref(args), layer, stream_handle(stream)),
           "adept_layer_step")


def embed(n, d_model, vocab, ids, table, h0, stream=None):
    _check(lib().adept_embed(dtype_code(table), n, d_model, vocab, ptr(ids), ptr(table), ptr(h0),
                             stream_handle(stream)), "adept_embed")


def final_logits(d_model, vocab, eps, h0, h1, exit_layer, rows, n_rows, max_rows, final_norm,
                 lm_head, x_norm, logits, stream=None):
    _check(lib().adept_final_logits(dtype_code(h0), d_model, vocab, eps, ptr(h0), ptr(h1),
                                    ptr(exit_layer), ptr(rows), ptr(n_rows), max_rows,
                                    ptr(final_norm), ptr(lm_head), ptr(x_norm), ptr(logits),
                                    stream_handle(stream)), "adept_final_logits")


def argmax(n, vocab, logits, out, stream=None):
    _check(lib().adept_argmax(n, vocab, ptr(logits), ptr(out), stream_handle(stream)),
           "adept_argmax")


def token_init(n_tok, n_layers, d_model, active, n_active, exit_layer, inertia=None, stream=None):
    _check(lib().adept_token_init(n_tok, n_layers, d_model, ptr(active), ptr(n_active),
                                  ptr(exit_layer), ptr(inertia), stream_handle(stream)),
           "adept_token_init")


def timing_enable(on=True):
    _check(lib().adept_timing_enable(1 if on else 0), "adept_timing_enable")


def timing_select(prefix=None):
    """Time only the launches whose kernel name starts with `prefix` (None: all)."""
    _check(lib().adept_timing_select(prefix.encode() if prefix else None),
           "adept_timing_select")


def timing_reset():
    lib().adept_timing_reset()


def encoder_workspace_bytes(args):
    return lib().adept_encoder_workspace_bytes(ctypes.byref(args))


def encoder_layer_step(args, layer, stream=None):
    _check(lib().adept_encoder_layer_step(ctypes.byref(args), layer, stream_handle(stream)),
           "adept_encoder_layer_step")


def encoder_embed(n, d_model, vocab, max_pos, eps, ids, pos, word_emb, pos_emb, type_emb, ln_g,
                  ln_b, out, stream=None):
    _check(lib().adept_encoder_embed(n, d_model, vocab, max_pos, eps, ptr(ids), ptr(pos),
                                     ptr(word_emb), ptr(pos_emb), ptr(type_emb), ptr(ln_g),
                                     ptr(ln_b), ptr(out), stream_handle(stream)),
           "adept_encoder_embed")


def classify_head(n_seq, seq_len, d_model, n_classes, h0, h1, exit_layer, w_cls, b_cls, logits,
                  stream=None):
    _check(lib().adept_classify_head(n_seq, seq_len, d_model, n_classes, ptr(h0), ptr(h1),
                                     ptr(exit_layer), ptr(w_cls), ptr(b_cls), ptr(logits),
                                     stream_handle(stream)), "adept_classify_head")


def timing_read():
    """{kernel name: (launches, total ms)} accumulated since the last reset."""
    L = lib()
    out = {}
    buf = ctypes.create_string_buffer(256)
    for i in range(L.adept_timing_count()):
        n, ms = _i64(0), ctypes.c_double(0.0)
        _check(L.adept_timing_get(i, buf, 256, ctypes.byref(n), ctypes.byref(ms)),
               "adept_timing_get")
        out[buf.value.decode()] = (int(n.value), float(ms.value))
    return out


def fold_gain(w, gain, stream=None):
    """In place: w[l][o][c] *= gain[l][c] for a stacked weight w [L, rows, cols]
    (or a [L, rows, cols] view with unit column stride) and gain [L, cols]."""
    L, rows, cols = w.shape
    assert w.stride(2) == 1 and gain.stride(-1) == 1 and gain.shape[-1] == cols
    if rows > 1:
        assert w.stride(1) == cols, "rows of each matrix must be contiguous"
    _check(lib().adept_fold_gain(dtype_code(w), L, rows, cols, ptr(w), w.stride(0), ptr(gain),
                                 gain.stride(0) if gain.dim() == 2 else 0, stream_handle(stream)),
           "adept_fold_gain")
