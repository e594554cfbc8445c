"""Independent reference for the oracle: HuggingFace transformers' Llama.

Builds a float64 `LlamaForCausalLM` whose weights are the synthetic weights of
a `synth` model shape (prompt-token embeddings appended to the vocabulary), so
the oracle's decoder, rotary embedding and tree attention can be checked
against a library implementation driven by a custom 4-D attention mask.
HF computes rotary angles in float32, so agreement is ~1e-6, not 1e-15."""
import numpy as np
import torch


def build_hf_llama(shape, W):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=shape.vocab + shape.n_prompt, hidden_size=shape.hidden,
                      intermediate_size=shape.ffn, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_base, max_position_embeddings=1 << 16,
                      tie_word_embeddings=False, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    hf = LlamaForCausalLM(cfg).double().eval()

    def f64(t):
        return t.detach().double().cpu()

    nq = shape.n_heads * shape.head_dim
    nk = shape.n_kv_heads * shape.head_dim
    sd = {
        "model.embed_tokens.weight": torch.cat([f64(W["tok_emb"]), f64(W["prompt_emb"])]),
        "model.norm.weight": f64(W["final_norm"]),
        "lm_head.weight": torch.cat([f64(W["lm_head"]),
                                     torch.zeros(shape.n_prompt, shape.hidden, dtype=torch.float64)]),
    }
    for l, lay in enumerate(W["layers"]):
        p = f"model.layers.{l}."
        qkv = f64(lay["w_qkv"])
        gu = f64(lay["w_gate_up"])
        sd[p + "self_attn.q_proj.weight"] = qkv[:nq]
        sd[p + "self_attn.k_proj.weight"] = qkv[nq:nq + nk]
        sd[p + "self_attn.v_proj.weight"] = qkv[nq + nk:]
        sd[p + "self_attn.o_proj.weight"] = f64(lay["w_o"])
        sd[p + "mlp.gate_proj.weight"] = gu[:shape.ffn]
        sd[p + "mlp.up_proj.weight"] = gu[shape.ffn:]
        sd[p + "mlp.down_proj.weight"] = f64(lay["w_down"])
        sd[p + "input_layernorm.weight"] = f64(lay["attn_norm"])
        sd[p + "post_attention_layernorm.weight"] = f64(lay["mlp_norm"])
    hf.load_state_dict(sd, strict=True)
    return hf


def hf_prefill(hf, ids):
    with torch.no_grad():
        out = hf(input_ids=torch.tensor(np.asarray(ids, np.int64)[None]), use_cache=True)
    return out.logits[0].numpy(), out.past_key_values


def hf_tree_logits(hf, pkv, L, ids, depth, anc, vocab):
    """Logits of tree nodes at positions L + depth under ancestor-only masking.
    `pkv` (the prefix cache) is copied, since HF appends to it in place."""
    import copy
    pkv = copy.deepcopy(pkv)
    T = len(ids)
    mask = torch.full((1, 1, T, L + T), float("-inf"), dtype=torch.float64)
    mask[0, 0, :, :L] = 0
    mask[0, 0, :, L:][torch.tensor(anc)] = 0
    with torch.no_grad():
        out = hf(input_ids=torch.tensor(np.asarray(ids, np.int64)[None]),
                 position_ids=torch.tensor((L + np.asarray(depth))[None]),
                 attention_mask=mask, past_key_values=pkv, use_cache=False)
    return out.logits[0, :, :vocab].numpy()
