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


# ---------------------------------------------------------------------------
# float64 throughout, and a bf16-storage variant
# ---------------------------------------------------------------------------
#
# Hugging Face computes RMSNorm and the rotary cos/sin tables in float32 even
# in a float64 model.  `hf_model_f64` keeps both in float64, so that the
# decoder agrees with the oracle to rounding order (~1e-12) instead of ~1e-5.
# `bf16_storage` then rounds, inside that decoder, every tensor a bf16
# implementation stores between two matrix products: the outputs of the three
# RMSNorms, v, q and k after the rotation, the softmax numerators before
# their product with V (the normaliser stays exact), the attention output
# before the o projection and the SwiGLU activation before the down
# projection.  These are hooks on the decoder's own modules; the oracle's
# forward pass is not involved.

import contextlib
import types


def _rms_f64(self, x):
    return self.weight * (x * torch.rsqrt(x.pow(2).mean(-1, keepdim=True) + self.variance_epsilon))


def hf_model_f64(cfg, W):
    from transformers.models.llama.modeling_llama import LlamaRMSNorm

    m = hf_model(cfg, W)
    for mod in m.modules():
        if isinstance(mod, LlamaRMSNorm):
            mod.forward = types.MethodType(_rms_f64, mod)
    dim, base = cfg.head_dim, float(cfg.rope_theta)

    def rotary_f64(self, x, position_ids):
        inv = 1.0 / (base ** (torch.arange(0, dim, 2, dtype=torch.float64) / dim))
        freqs = position_ids[..., None].to(torch.float64) * inv
        emb = torch.cat((freqs, freqs), dim=-1)
        return emb.cos(), emb.sin()

    m.model.rotary_emb.forward = types.MethodType(rotary_f64, m.model.rotary_emb)
    return m


STORAGE_POINTS = ("norm", "v", "qk", "numerators", "attn_out", "act")


@contextlib.contextmanager
def bf16_storage(model, dtype=torch.bfloat16, skip=()):
    """Round the storage points listed in STORAGE_POINTS (minus ``skip``) to
    ``dtype`` while the context is open."""
    from transformers.modeling_utils import ALL_ATTENTION_FUNCTIONS
    from transformers.models.llama import modeling_llama as ml

    def rnd(t):
        return t.to(dtype).to(torch.float64)

    on = set(STORAGE_POINTS) - set(skip)
    handles = []
    out_hook = lambda mod, args, out: rnd(out)          # noqa: E731
    in_hook = lambda mod, args: (rnd(args[0]),)         # noqa: E731
    for layer in model.model.layers:
        if "norm" in on:
            handles.append(layer.input_layernorm.register_forward_hook(out_hook))
            handles.append(layer.post_attention_layernorm.register_forward_hook(out_hook))
        if "v" in on:
            handles.append(layer.self_attn.v_proj.register_forward_hook(out_hook))
        if "attn_out" in on:
            handles.append(layer.self_attn.o_proj.register_forward_pre_hook(in_hook))
        if "act" in on:
            handles.append(layer.mlp.down_proj.register_forward_pre_hook(in_hook))
    if "norm" in on:
        handles.append(model.model.norm.register_forward_hook(out_hook))

    orig_rope = ml.apply_rotary_pos_emb
    if "qk" in on:
        def rope_rounded(q, k, cos, sin, unsqueeze_dim=1):
            qe, ke = orig_rope(q, k, cos, sin, unsqueeze_dim)
            return rnd(qe), rnd(ke)
        ml.apply_rotary_pos_emb = rope_rounded

    def attn_rounded_numerators(module, query, key, value, attention_mask, scaling, dropout=0.0,
                                **kwargs):
        ks = ml.repeat_kv(key, module.num_key_value_groups)
        vs = ml.repeat_kv(value, module.num_key_value_groups)
        s = torch.matmul(query, ks.transpose(2, 3)) * scaling
        if attention_mask is not None:
            s = s + attention_mask
        else:   # the decoder hands custom attention functions no mask: causal
            lq, lk = s.shape[-2], s.shape[-1]
            causal = torch.ones(lq, lk, dtype=torch.bool).tril(lk - lq)
            s = s.masked_fill(~causal, float("-inf"))
        e = torch.exp(s - s.amax(dim=-1, keepdim=True))
        num = rnd(e) if "numerators" in on else e
        out = torch.matmul(num, vs) / e.sum(dim=-1, keepdim=True)
        return out.transpose(1, 2).contiguous(), None

    name = "oracle_pin_bf16_numerators"
    ALL_ATTENTION_FUNCTIONS[name] = attn_rounded_numerators
    prev_impl = model.config._attn_implementation
    model.config._attn_implementation = name
    try:
        yield model
    finally:
        model.config._attn_implementation = prev_impl
        ml.apply_rotary_pos_emb = orig_rope
        for h in handles:
            h.remove()
