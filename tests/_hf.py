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


def bf16_round_f64(t: torch.Tensor) -> torch.Tensor:
    """Round float64 values to the nearest bfloat16 (ties to even) in ONE
    rounding, returned as float64.  torch converts float64 to bfloat16
    through float32 (two roundings); the two differ only where the float32
    value lands exactly halfway between two bfloat16 values although the
    double did not, and there the side the double lay on decides.  Finite,
    normal-range inputs only (what the tests feed it)."""
    t = t.to(torch.float64)
    f = t.to(torch.float32)
    out = f.to(torch.bfloat16).to(torch.float64)
    bits = f.view(torch.int32)
    tie = ((bits & 0xFFFF) == 0x8000) & (f.to(torch.float64) != t)
    if bool(tie.any()):
        lo = (bits & ~0xFFFF).view(torch.float32).to(torch.float64)   # toward zero
        hi = (bits + 0x8000).view(torch.float32).to(torch.float64)    # away from zero
        away = t.abs() > f.to(torch.float64).abs()
        out = torch.where(tie, torch.where(away, hi, lo), out)
    return out


def hf_model_exact(cfg: dict, layers: list, keep: list):
    """hf_model with float64 arithmetic end to end: rotary angles computed in
    float64 (HF computes them in float32), RMSNorm in float64 (HF's casts to
    float32) and attention through torch's scaled_dot_product_attention,
    whose softmax stays in float64 (HF's eager attention takes the softmax
    in float32)."""
    m = hf_model(cfg, layers, keep)
    eps = float(cfg["rms_eps"])

    def rms64(norm):
        def fwd(x):
            return norm.weight * (x * torch.rsqrt(x.pow(2).mean(-1, keepdim=True) + eps))
        return fwd

    for blk in m.layers:
        blk.input_layernorm.forward = rms64(blk.input_layernorm)
        blk.post_attention_layernorm.forward = rms64(blk.post_attention_layernorm)
    m.config._attn_implementation = "sdpa"
    for blk in m.layers:
        blk.self_attn.config._attn_implementation = "sdpa"
    hd, theta = cfg["head_dim"], float(cfg["rope_theta"])
    inv = 1.0 / (theta ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))

    def rope64(x, position_ids):
        ang = position_ids[..., None].to(torch.float64) * inv
        emb = torch.cat([ang, ang], dim=-1)
        return emb.cos(), emb.sin()

    m.rotary_emb.forward = rope64
    return m


def hf_decode_rounded_cache(model, x: np.ndarray, round_kv=bf16_round_f64):
    """Token-by-token decode of x [T][d] through a KV cache whose new K/V
    rows (after the rotary embedding) are rounded by round_kv before any
    attention reads them, as a bf16 cache stores them.  Returns the last
    block's outputs [T][d] and the cache (per block: K, V [n_kv][T][hd])."""
    from transformers import DynamicCache

    class RoundedCache(DynamicCache):
        def update(self, key_states, value_states, layer_idx, *a, **kw):
            return super().update(round_kv(key_states), round_kv(value_states), layer_idx,
                                  *a, **kw)

    cache = RoundedCache()
    outs = []
    with torch.no_grad():
        for t in range(x.shape[0]):
            xt = torch.from_numpy(x[t:t + 1].astype(np.float64))[None]
            pid = torch.tensor([[t]])
            out = model(inputs_embeds=xt, position_ids=pid, past_key_values=cache,
                        use_cache=True, cache_position=torch.tensor([t]))
            outs.append(out.last_hidden_state[0, 0].numpy())
    kv = [(cache.layers[i].keys[0].numpy(), cache.layers[i].values[0].numpy())
          for i in range(len(model.layers))]
    return np.array(outs), kv
