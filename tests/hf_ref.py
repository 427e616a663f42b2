"""Independent reference for the oracle's decoder: the Hugging Face
``transformers`` Llama implementation run on the CPU in float64.

Used only by the CPU pin tests.  The oracle does not import it.
"""
import numpy as np
import torch


def hf_llama(shape, weights):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
        rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta,
        max_position_embeddings=4096, tie_word_embeddings=False,
        attention_bias=False, mlp_bias=False, hidden_act="silu")
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).double().eval()
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64).copy())
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(weights["tok_emb"]))
        for l, lw in enumerate(weights["layers"]):
            L = m.model.layers[l]
            L.self_attn.q_proj.weight.copy_(t(lw["wq"]))
            L.self_attn.k_proj.weight.copy_(t(lw["wk"]))
            L.self_attn.v_proj.weight.copy_(t(lw["wv"]))
            L.self_attn.o_proj.weight.copy_(t(lw["wo"]))
            L.mlp.gate_proj.weight.copy_(t(lw["w_gate"]))
            L.mlp.up_proj.weight.copy_(t(lw["w_up"]))
            L.mlp.down_proj.weight.copy_(t(lw["w_down"]))
            L.input_layernorm.weight.copy_(t(lw["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(t(lw["mlp_norm"]))
        m.model.norm.weight.copy_(t(weights["final_norm"]))
        m.lm_head.weight.copy_(t(weights["lm_head"]))
    return m


def hf_logits(model, tokens):
    with torch.no_grad():
        out = model(torch.tensor([list(map(int, tokens))], dtype=torch.long))
    return out.logits[0].numpy()


def hf_greedy(model, prompt, n_new):
    """Plain greedy decoding by repeated full forwards (argmax, lowest id)."""
    seq = [int(t) for t in prompt]
    for _ in range(n_new):
        z = hf_logits(model, seq)[-1]
        seq.append(int(np.argmax(z)))
    return seq[len(prompt):]


def hf_hidden(model, tokens):
    """Final-normed hidden states [T, D] (the base model's output, after the
    last RMSNorm)."""
    with torch.no_grad():
        out = model.model(torch.tensor([list(map(int, tokens))], dtype=torch.long))
    return out.last_hidden_state[0].numpy()
