"""Seeded synthetic inputs for BUDDY's routed decode step.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic.  The same tensors feed the GPU library and the CPU
oracle, so both sides see identical inputs.

The paper measures decode speed on Alpaca and SAMSum prompts with trained
Llama/Qwen weights (Sec. 5, speed analysis); neither is available here, so
these generators stand in for them with random-init models of the same
shapes and random KV caches of the stated context lengths.
"""
from __future__ import annotations

import dataclasses

import torch

# Model shapes.  Llama-3-8B, Qwen2.5-7B and a Llama-1-13B-sized MHA model are
# the paper's backbones (Sec. 5 settings, App. "LLM versions"); the tiny model
# is a parity-sized decoder with the same structure.
SHAPES = {
    "tiny": dict(n_layers=8, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64,
                 d_ffn=688, dm_hidden=128, dm_act="gelu", rope_theta=1e4, rms_eps=1e-5),
    "llama3_8b": dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                      d_ffn=14336, dm_hidden=512, dm_act="silu", rope_theta=5e5, rms_eps=1e-5),
    "qwen2_7b": dict(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
                     d_ffn=18944, dm_hidden=512, dm_act="silu", rope_theta=1e6, rms_eps=1e-6),
    "mha_13b": dict(n_layers=40, d_model=5120, n_heads=40, n_kv_heads=40, head_dim=128,
                    d_ffn=13824, dm_hidden=512, dm_act="silu", rope_theta=1e4, rms_eps=1e-6),
}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: str
    dtype: str          # storage of weights and KV: "f32" or "bf16"
    batch: int
    ctx: int            # cached positions before the first timed step
    steps: int
    budgets: tuple      # k values; one per run, or the set drawn from per sequence
    mixed: bool         # True: k_b drawn uniformly from `budgets` per sequence
    omega: float        # prior weight in the score fusion (0 = no prior)

    @property
    def max_ctx(self) -> int:
        return self.ctx + self.steps


WORKLOADS = {
    "tiny_b4_prompt64": Workload("tiny_b4_prompt64", "tiny", "f32", 4, 64, 16, (3,), False, 0.0),
    "llama3_8b_b1_ctx2048": Workload("llama3_8b_b1_ctx2048", "llama3_8b", "bf16", 1, 2048, 128,
                                     (15, 22, 30), False, 0.1),
    "llama3_8b_b32_ctx4096_mixed": Workload("llama3_8b_b32_ctx4096_mixed", "llama3_8b", "bf16",
                                            32, 4096, 128, (12, 18, 24, 30), True, 0.1),
    "qwen2_7b_b64_ctx8192": Workload("qwen2_7b_b64_ctx8192", "qwen2_7b", "bf16", 64, 8192, 64,
                                     (18,), False, 0.1),
    "mha_13b_b96_ctx2048_mixed": Workload("mha_13b_b96_ctx2048_mixed", "mha_13b", "bf16", 96,
                                          2048, 64, (19, 28, 38), True, 0.1),
}


def context_dim(cfg: dict) -> int:
    """Number of router-context inputs (the Decision Module's first-layer
    width) for the configured variant: 'kv' pools K and V side by side, 'k',
    'v' and 'k+v' one head-major vector; the newest hidden state follows."""
    n = cfg["n_kv_heads"] * cfg["head_dim"]
    return (2 * n if cfg.get("router_ctx", "kv") == "kv" else n) + cfg["d_model"]


def n_mid(cfg: dict) -> int:
    """Routable blocks S..L-2 for start layer S (default 1): L - 1 - S."""
    return cfg["n_layers"] - 1 - int(cfg.get("start_layer", 1))


def model_config(shape: str | dict, dtype: str, max_ctx: int) -> dict:
    s = SHAPES[shape] if isinstance(shape, str) else shape
    c = dict(s)
    c["dtype"] = dtype
    c["max_ctx"] = int(max_ctx)
    return c


def _tdtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def _normal(shape, std, mean, gen, device, dtype):
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(mean=mean, std=std, generator=gen)
    return t.to(_tdtype(dtype))


def model_weights(cfg: dict, seed: int, device="cpu", omega: float = 0.1,
                  std: float = 0.02) -> dict:
    """Random-init weights: linear and Decision Module weights and biases
    N(0, std); RMSNorm gains 1 + N(0, std); prior N(0, 1) (a stand-in for an
    already normalised prior).  Row-major [out][in] layouts:
    wqkv rows q|k|v, wgate_up rows gate|up."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    d, nq, nkv, hd, f = (cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                         cfg["head_dim"], cfg["d_ffn"])
    dt = cfg["dtype"]
    layers = []
    for _ in range(cfg["n_layers"]):
        layers.append(dict(
            attn_norm=_normal((d,), std, 1.0, gen, device, dt),
            wqkv=_normal(((nq + 2 * nkv) * hd, d), std, 0.0, gen, device, dt),
            wo=_normal((d, nq * hd), std, 0.0, gen, device, dt),
            mlp_norm=_normal((d,), std, 1.0, gen, device, dt),
            wgate_up=_normal((2 * f, d), std, 0.0, gen, device, dt),
            wdown=_normal((d, f), std, 0.0, gen, device, dt),
        ))
    H, Lm = cfg["dm_hidden"], n_mid(cfg)
    din = context_dim(cfg)
    dm = dict(
        w1=_normal((H, din), std, 0.0, gen, device, dt),
        b1=_normal((H,), std, 0.0, gen, device, dt),
        w2=_normal((Lm, H), std, 0.0, gen, device, dt),
        b2=_normal((Lm,), std, 0.0, gen, device, dt),
        prior=_normal((Lm,), 1.0, 0.0, gen, device, "f32") if omega else None,
        omega=float(omega),
    )
    return dict(layers=layers, dm=dm)


def predictor_weights(cfg: dict, hidden: int, seed: int, device="cpu", std: float = 0.02) -> dict:
    """Random-init Budget Predictor head: w1 [hidden][din], b1, w2 [L_mid][hidden],
    b2, all N(0, std) in the storage dtype (no trained predictor exists)."""
    gen = torch.Generator(device=device).manual_seed(seed)
    dt, Lm = cfg["dtype"], n_mid(cfg)
    return dict(
        w1=_normal((hidden, context_dim(cfg)), std, 0.0, gen, device, dt),
        b1=_normal((hidden,), std, 0.0, gen, device, dt),
        w2=_normal((Lm, hidden), std, 0.0, gen, device, dt),
        b2=_normal((Lm,), std, 0.0, gen, device, dt),
    )


def kv_cache(cfg: dict, batch: int, ctx: int, seed: int, device="cpu",
             fill_std: float = 1.0) -> tuple:
    """K and V caches [L][B][n_kv][max_ctx][hd]; positions < ctx hold
    N(0, fill_std) values, the rest zero."""
    L, nkv, hd, T = cfg["n_layers"], cfg["n_kv_heads"], cfg["head_dim"], cfg["max_ctx"]
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    out = []
    for _ in range(2):
        t = torch.zeros((L, batch, nkv, T, hd), dtype=_tdtype(cfg["dtype"]), device=device)
        if ctx > 0:
            for l in range(L):   # filled in place, one layer at a time
                t[l, :, :, :ctx, :].normal_(mean=0.0, std=fill_std, generator=gen)
        out.append(t)
    return tuple(out)


def hidden_inputs(n: int, d: int, seed: int, device="cpu") -> torch.Tensor:
    """n hidden vectors N(0, 1), float32 [n][d]."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    t = torch.empty((n, d), dtype=torch.float32, device=device)
    t.normal_(generator=gen)
    return t


def budgets(w: Workload, seed: int, k: int | None = None) -> list:
    """Per-sequence k: a fixed k for every sequence, or (mixed workloads)
    i.i.d. uniform over the workload's budget set."""
    if not w.mixed:
        return [int(k if k is not None else w.budgets[0])] * w.batch
    gen = torch.Generator()
    gen.manual_seed(seed)
    idx = torch.randint(0, len(w.budgets), (w.batch,), generator=gen)
    return [int(w.budgets[i]) for i in idx]


def storage_numpy(t: torch.Tensor):
    """Host numpy view of a storage tensor: bf16 -> uint16 bits, fp32 as is."""
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    return t.numpy()
