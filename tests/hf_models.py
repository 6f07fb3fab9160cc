"""Hugging Face reference models built from the seeded weights (fp64, CPU).

Used only by the oracle pins: the transformers library's Llama and BERT
implementations are an independent statement of the base models' layers."""
import numpy as np
import torch


def _t(x):
    return torch.from_numpy(np.asarray(x, np.float64).copy())


def llama(shape, weights, n_layers=None):
    from transformers import LlamaConfig, LlamaForCausalLM
    n_layers = shape.n_layers if n_layers is None else n_layers
    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model,
                      intermediate_size=shape.d_ff, num_hidden_layers=n_layers,
                      num_attention_heads=shape.n_heads, num_key_value_heads=shape.n_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_theta, max_position_embeddings=4096,
                      tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                      attn_implementation="eager")
    m = LlamaForCausalLM(cfg).double().eval()
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(_t(weights["embed"]))
        m.model.norm.weight.copy_(_t(weights["final_norm"]))
        m.lm_head.weight.copy_(_t(weights["lm_head"]))
        for i in range(n_layers):
            lw, L = weights["layers"][i], m.model.layers[i]
            L.input_layernorm.weight.copy_(_t(lw["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(_t(lw["ffn_norm"]))
            L.self_attn.q_proj.weight.copy_(_t(lw["wq"]))
            L.self_attn.k_proj.weight.copy_(_t(lw["wk"]))
            L.self_attn.v_proj.weight.copy_(_t(lw["wv"]))
            L.self_attn.o_proj.weight.copy_(_t(lw["wo"]))
            L.mlp.gate_proj.weight.copy_(_t(lw["w_gate"]))
            L.mlp.up_proj.weight.copy_(_t(lw["w_up"]))
            L.mlp.down_proj.weight.copy_(_t(lw["w_down"]))
    return m


def bert(shape, weights, n_layers=None):
    from transformers import BertConfig, BertModel
    n_layers = shape.n_layers if n_layers is None else n_layers
    cfg = BertConfig(vocab_size=shape.vocab, hidden_size=shape.d_model,
                     num_hidden_layers=n_layers, num_attention_heads=shape.n_heads,
                     intermediate_size=shape.d_ff, hidden_act="gelu",
                     max_position_embeddings=shape.max_pos, type_vocab_size=1,
                     layer_norm_eps=shape.ln_eps, hidden_dropout_prob=0.0,
                     attention_probs_dropout_prob=0.0, attn_implementation="eager")
    m = BertModel(cfg, add_pooling_layer=False).double().eval()
    with torch.no_grad():
        e = m.embeddings
        e.word_embeddings.weight.copy_(_t(weights["word_embed"]))
        e.position_embeddings.weight.copy_(_t(weights["pos_embed"]))
        e.token_type_embeddings.weight.copy_(_t(weights["type_embed"])[None, :])
        e.LayerNorm.weight.copy_(_t(weights["embed_ln_g"]))
        e.LayerNorm.bias.copy_(_t(weights["embed_ln_b"]))
        for i in range(n_layers):
            lw, L = weights["layers"][i], m.encoder.layer[i]
            a = L.attention
            for mod, w, b in ((a.self.query, "wq", "bq"), (a.self.key, "wk", "bk"),
                              (a.self.value, "wv", "bv"), (a.output.dense, "wo", "bo"),
                              (L.intermediate.dense, "w_in", "b_in"),
                              (L.output.dense, "w_out", "b_out")):
                mod.weight.copy_(_t(lw[w]))
                mod.bias.copy_(_t(lw[b]))
            a.output.LayerNorm.weight.copy_(_t(lw["ln1_g"]))
            a.output.LayerNorm.bias.copy_(_t(lw["ln1_b"]))
            L.output.LayerNorm.weight.copy_(_t(lw["ln2_g"]))
            L.output.LayerNorm.bias.copy_(_t(lw["ln2_b"]))
    return m


def gpt2(shape, weights, n_layers=None):
    """transformers' GPT2LMHeadModel (tanh GELU, LayerNorm with bias, learned
    positions, head tied to the token embedding) with the seeded weights;
    Conv1D layers hold their weight as [in, out], the transpose of ours."""
    from transformers import GPT2Config, GPT2LMHeadModel
    n_layers = shape.n_layers if n_layers is None else n_layers
    cfg = GPT2Config(vocab_size=shape.vocab, n_positions=shape.max_pos, n_embd=shape.d_model,
                     n_layer=n_layers, n_head=shape.n_heads, n_inner=shape.d_ff,
                     activation_function="gelu_new", resid_pdrop=0.0, embd_pdrop=0.0,
                     attn_pdrop=0.0, layer_norm_epsilon=shape.ln_eps, tie_word_embeddings=True,
                     attn_implementation="eager")
    m = GPT2LMHeadModel(cfg).double().eval()
    with torch.no_grad():
        m.transformer.wte.weight.copy_(_t(weights["embed"]))
        m.transformer.wpe.weight.copy_(_t(weights["pos_embed"]))
        m.transformer.ln_f.weight.copy_(_t(weights["final_ln_g"]))
        m.transformer.ln_f.bias.copy_(_t(weights["final_ln_b"]))
        for i in range(n_layers):
            lw, L = weights["layers"][i], m.transformer.h[i]
            L.ln_1.weight.copy_(_t(lw["ln1_g"]))
            L.ln_1.bias.copy_(_t(lw["ln1_b"]))
            L.ln_2.weight.copy_(_t(lw["ln2_g"]))
            L.ln_2.bias.copy_(_t(lw["ln2_b"]))
            wqkv = np.concatenate([lw["wq"], lw["wk"], lw["wv"]], axis=0)
            L.attn.c_attn.weight.copy_(_t(wqkv.T))
            L.attn.c_attn.bias.copy_(_t(np.concatenate([lw["bq"], lw["bk"], lw["bv"]])))
            L.attn.c_proj.weight.copy_(_t(np.asarray(lw["wo"]).T))
            L.attn.c_proj.bias.copy_(_t(lw["bo"]))
            L.mlp.c_fc.weight.copy_(_t(np.asarray(lw["w_fc"]).T))
            L.mlp.c_fc.bias.copy_(_t(lw["b_fc"]))
            L.mlp.c_proj.weight.copy_(_t(np.asarray(lw["w_proj"]).T))
            L.mlp.c_proj.bias.copy_(_t(lw["b_proj"]))
    return m
