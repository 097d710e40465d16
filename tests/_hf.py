"""Dense reference forward with Hugging Face's Llama implementation.

Used only to pin the oracle: with every routable layer selected, a routed
decode over a sequence must equal a dense causal forward of the same stack
(Sec. 3.1 Eq. 1 with M = 1 everywhere), and a fixed route must equal the
dense forward of the sub-model made of the selected blocks.
"""
import numpy as np
import torch


def _f64(a):
    if a.dtype == np.uint16:
        return torch.from_numpy((a.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    return torch.from_numpy(a.astype(np.float64))


def hf_model(cfg: dict, layers: list, keep: list):
    """LlamaModel (float64, eager attention, no final norm) made of the blocks
    listed in `keep`, with weights taken from the storage arrays `layers`."""
    from transformers import LlamaConfig, LlamaModel
    hd, nq, nkv, d, f = (cfg["head_dim"], cfg["n_heads"], cfg["n_kv_heads"],
                         cfg["d_model"], cfg["d_ffn"])
    hc = LlamaConfig(hidden_size=d, intermediate_size=f, num_hidden_layers=len(keep),
                     num_attention_heads=nq, num_key_value_heads=nkv, head_dim=hd,
                     rms_norm_eps=cfg["rms_eps"], rope_theta=cfg["rope_theta"],
                     vocab_size=8, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096)
    hc._attn_implementation = "eager"
    m = LlamaModel(hc).double().eval()
    m.norm = torch.nn.Identity()
    with torch.no_grad():
        for j, li in enumerate(keep):
            w = layers[li]
            blk = m.layers[j]
            wqkv = _f64(w["wqkv"])
            blk.self_attn.q_proj.weight.copy_(wqkv[: nq * hd])
            blk.self_attn.k_proj.weight.copy_(wqkv[nq * hd:(nq + nkv) * hd])
            blk.self_attn.v_proj.weight.copy_(wqkv[(nq + nkv) * hd:])
            blk.self_attn.o_proj.weight.copy_(_f64(w["wo"]))
            gu = _f64(w["wgate_up"])
            blk.mlp.gate_proj.weight.copy_(gu[:f])
            blk.mlp.up_proj.weight.copy_(gu[f:])
            blk.mlp.down_proj.weight.copy_(_f64(w["wdown"]))
            blk.input_layernorm.weight.copy_(_f64(w["attn_norm"]))
            blk.post_attention_layernorm.weight.copy_(_f64(w["mlp_norm"]))
    return m


def hf_forward(model, x: np.ndarray) -> np.ndarray:
    """Dense causal forward over x [T][d]; returns the last block's output [T][d]."""
    with torch.no_grad():
        out = model(inputs_embeds=torch.from_numpy(x.astype(np.float64))[None])
    return out.last_hidden_state[0].numpy()


def hf_routed_masked(model, x: np.ndarray, routes: np.ndarray) -> np.ndarray:
    """Per-token routes with skipped-KV masking, computed without a KV cache:
    block l (of the full stack `model`) runs causally over the subsequence of
    tokens that execute it, each at its own position (rotary angles of the
    original positions).  Block 0 and the last block run for every token;
    routes [T][L-2] select the others.  Decoding is causal per block, so this
    equals a token-by-token decode in which each block attends only to the
    positions at which it ran.  Returns the last block's output [T][d]."""
    T, L = x.shape[0], len(model.layers)
    run = np.ones((T, L), dtype=bool)
    run[:, 1:L - 1] = routes.astype(bool)
    h = torch.from_numpy(x.astype(np.float64)).clone()
    with torch.no_grad():
        for li in range(L):
            idx = np.nonzero(run[:, li])[0]
            if idx.size == 0:
                continue
            sub = h[idx][None]
            pid = torch.from_numpy(idx.astype(np.int64))[None]
            cos_sin = model.rotary_emb(sub, pid)
            n = idx.size
            mask = torch.full((n, n), float("-inf"), dtype=torch.float64).triu(1)[None, None]
            out = model.layers[li](sub, attention_mask=mask, position_ids=pid,
                                   position_embeddings=cos_sin)
            out = out[0] if isinstance(out, tuple) else out
            h[idx] = out[0]
    return h.numpy()
