"""Hugging Face's Llama implementation as an independent reference for the oracle.

The paper implements prepacking on top of Hugging Face Transformers models
(sections 4 and 4.2): a custom attention mask plus position ids.  Running the
same weights through Hugging Face's own Llama code, in float64 on the CPU, is
therefore an independent check of the oracle's decoder, of the independent
mask and restart positions, and of the full-batching baseline.  Test helper only.
"""
import numpy as np
import torch


def build(shape, weights):
    from transformers import LlamaConfig, LlamaModel
    cfg = LlamaConfig(hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
                      num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
                      num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                      vocab_size=shape.vocab, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_theta, attn_implementation="eager")
    model = LlamaModel(cfg).double().eval()
    sd = {"embed_tokens.weight": weights["embed"], "norm.weight": weights["final_norm"]}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj",
             "wd": "mlp.down_proj", "attn_norm": "input_layernorm",
             "mlp_norm": "post_attention_layernorm"}
    for i, L in enumerate(weights["layers"][: shape.n_layers]):
        for key, name in names.items():
            sd[f"layers.{i}.{name}.weight"] = L[key]
    model.load_state_dict({k: torch.from_numpy(np.asarray(v, dtype=np.float64)) for k, v in sd.items()})
    return model


def last_logits(shape, weights, lm_head, ids):
    """Hugging Face's causal LM (LlamaForCausalLM: the decoder, its final norm and the LM
    head) on one prompt; the float64 logits at the prompt's last position, [vocab]."""
    from transformers import LlamaForCausalLM
    base = build(shape, weights)
    lm = LlamaForCausalLM(base.config).double().eval()
    lm.model = base
    lm.lm_head.weight.data = torch.from_numpy(np.asarray(lm_head, dtype=np.float64))
    with torch.no_grad():
        out = lm(input_ids=torch.as_tensor(ids, dtype=torch.long)[None])
    return out.logits[0, -1].numpy()


def run(model, ids, attention_mask=None, position_ids=None):
    """Returns (hidden [b, n, d], [K_l [b, n, Hkv*D]], [V_l ...]) as numpy float64."""
    with torch.no_grad():
        out = model(input_ids=torch.as_tensor(ids, dtype=torch.long),
                    attention_mask=attention_mask,
                    position_ids=None if position_ids is None else torch.as_tensor(position_ids, dtype=torch.long),
                    use_cache=True)
    h = out.last_hidden_state.numpy()
    ks, vs = [], []
    for layer in out.past_key_values.layers:
        k = layer.keys.numpy()            # [b, Hkv, n, D]
        v = layer.values.numpy()
        b, hk, n, d = k.shape
        ks.append(k.transpose(0, 2, 1, 3).reshape(b, n, hk * d))
        vs.append(v.transpose(0, 2, 1, 3).reshape(b, n, hk * d))
    return h, ks, vs


def additive_mask(allowed):
    """Boolean [b, n, n] -> additive float64 [b, 1, n, n]; a query with no allowed key is
    let see itself (its output is discarded) so that the reference stays finite."""
    allowed = np.array(allowed, dtype=bool)
    for b in range(allowed.shape[0]):
        empty = ~allowed[b].any(axis=1)
        idx = np.nonzero(empty)[0]
        allowed[b, idx, idx] = True
    m = torch.zeros(allowed.shape, dtype=torch.float64)
    m[~torch.from_numpy(allowed)] = torch.finfo(torch.float64).min
    return m[:, None]


def greedy_generate(shape, weights, lm_head, ids, n_tokens):
    """Hugging Face's greedy generate (its own incremental decoding with a KV cache) on one
    prompt: the n_tokens new ids, and per layer the cached K, V of the positions after the
    prompt ([n_tokens - 1, Hkv*D]: the last token is chosen but never fed)."""
    from transformers import GenerationConfig, LlamaForCausalLM
    base = build(shape, weights)
    lm = LlamaForCausalLM(base.config).double().eval()
    lm.model = base
    lm.lm_head.weight.data = torch.from_numpy(np.asarray(lm_head, dtype=np.float64))
    gc = GenerationConfig(max_new_tokens=n_tokens, min_new_tokens=n_tokens, do_sample=False, num_beams=1,
                          eos_token_id=None, pad_token_id=0, bos_token_id=None)
    gc.return_dict_in_generate, gc.use_cache = True, True
    ids_t = torch.as_tensor(ids, dtype=torch.long)[None]
    with torch.no_grad():   # an explicit mask: otherwise ids equal to the pad id would be masked out
        out = lm.generate(input_ids=ids_t, attention_mask=torch.ones_like(ids_t), generation_config=gc)
    l = len(ids)
    new = out.sequences[0, l:].numpy()
    ks, vs = [], []
    for layer in out.past_key_values.layers:
        k = layer.keys.numpy()[0]        # [Hkv, n, D]
        v = layer.values.numpy()[0]
        hk, n, d = k.shape
        ks.append(k.transpose(1, 0, 2).reshape(n, hk * d)[l:])
        vs.append(v.transpose(1, 0, 2).reshape(n, hk * d)[l:])
    return new, ks, vs
