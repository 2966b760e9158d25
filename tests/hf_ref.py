"""An independent Llama decoder (Hugging Face ``LlamaForCausalLM``) in float64,
loaded with the same weights the oracle sees.  Used only to pin the oracle:
a branch of a draft tree, decoded on its own after the prompt, must give the
same logits as the oracle's tree evaluation."""

import torch


def hf_model(cfg, W):
    from transformers import LlamaConfig, LlamaForCausalLM

    c = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.ffn,
                    num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                    num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                    rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                    tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                    max_position_embeddings=8192)
    c._attn_implementation = "eager"
    m = LlamaForCausalLM(c).to(torch.float64).eval()
    sd = {"model.embed_tokens.weight": W["tok_embed"], "model.norm.weight": W["final_norm"],
          "lm_head.weight": W["lm_head"]}
    names = {"attn_norm": "input_layernorm", "ffn_norm": "post_attention_layernorm",
             "wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
             "w_down": "mlp.down_proj"}
    for l, lw in enumerate(W["layers"]):
        for k, v in lw.items():
            sd[f"model.layers.{l}.{names[k]}.weight"] = v
    sd = {k: v.detach().to(torch.float64) for k, v in sd.items()}
    missing, unexpected = m.load_state_dict(sd, strict=False)
    missing = [k for k in missing if "rotary" not in k]
    assert not missing and not unexpected, (missing, unexpected)
    return m


@torch.no_grad()
def hf_logits(model, seq):
    """Next-token logits after every prefix of ``seq`` (float64 [len, V])."""
    ids = torch.tensor([list(seq)], dtype=torch.int64)
    return model(input_ids=ids, use_cache=False).logits[0]


@torch.no_grad()
def hf_greedy(model, prompt, n):
    """Plain autoregressive greedy decoding: ``n`` new tokens after ``prompt``."""
    seq = list(prompt)
    out = []
    for _ in range(n):
        t = int(torch.argmax(hf_logits(model, seq)[-1]))
        out.append(t)
        seq.append(t)
    return out
