"""Analytic cost model of the routed decode step (host logic).

- Budget to layer count: k = round(b L) - 2 (Sec. 4.2.1, Eq. 2); the App. C.2
  variant k = b L - I clamped to [1, L - I].
- FLOP model of App. C.2: F_DM = 2BTdr + 2BTr(L - I),
  F_layer = 8Td^2 + 4T^2 d + 4T d d_c, F_model(b) = b L F_layer and
  rho(b) = F_DM / F_model(b).
- Algorithmic bytes of one decode step, which the benchmark divides by the
  measured step time to get the fraction of the HBM roofline: the weights of
  every block some sequence executes (read once per step), the KV rows each
  executed (sequence, block) pair attends, the first-layer KV scan of the
  router context, the Decision Module weights, and the new K/V rows written.
"""
from __future__ import annotations

import math


def budget_to_k(b: float, n_layers: int, clamp: bool = False, ignored: int = 2) -> int:
    """Eq. 2: k = round(b L) - 2, rounding halves away from zero.  With
    clamp=True the App. C.2 form k = b L - I limited to [1, L - I]."""
    if not (0.0 < b <= 1.0):
        raise ValueError("budget must lie in (0, 1]")
    k = int(math.floor(b * n_layers + 0.5)) - ignored
    if clamp:
        k = min(max(k, 1), n_layers - ignored)
    return max(k, 0)


def k_to_budget(k: int, n_layers: int) -> float:
    """Budget Predictor inverse map b = (k + 2) / L (Sec. 4.4)."""
    return (k + 2) / n_layers


def dm_flops(B: int, T: int, d: int, r: int, L: int, I: int = 2) -> int:
    return 2 * B * T * d * r + 2 * B * T * r * (L - I)


def layer_flops(T: int, d: int, d_c: int) -> int:
    return 8 * T * d * d + 4 * T * T * d + 4 * T * d * d_c


def model_flops(b: float, L: int, T: int, d: int, d_c: int) -> float:
    return b * L * layer_flops(T, d, d_c)


def dm_overhead(b: float, B: int, T: int, d: int, d_c: int, r: int, L: int, I: int = 2) -> float:
    return dm_flops(B, T, d, r, L, I) / model_flops(b, L, T, d, d_c)


# ------------------------------------------------------------ bytes per step

def _s(dtype: str) -> int:
    return 2 if dtype == "bf16" else 4


def layer_weight_bytes(cfg: dict) -> int:
    d, nq, nkv, hd, f = (cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                         cfg["head_dim"], cfg["d_ffn"])
    elems = d * (nq + 2 * nkv) * hd + nq * hd * d + 3 * d * f + 2 * d
    return elems * _s(cfg["dtype"])


def dm_weight_bytes(cfg: dict) -> int:
    H, Lm = cfg["dm_hidden"], cfg["n_layers"] - 1 - int(cfg.get("start_layer", 1))
    n = cfg["n_kv_heads"] * cfg["head_dim"]
    din = (2 * n if cfg.get("router_ctx", "kv") == "kv" else n) + cfg["d_model"]
    return (H * din + H + Lm * H + Lm) * _s(cfg["dtype"])


def step_bytes(cfg: dict, masks, positions, running_pool: bool = False,
               pool_fused: bool = False) -> dict:
    """Algorithmic bytes of one step given the realised per-sequence masks
    (each a sequence of L_mid zeros/ones for blocks S..L-2) and the positions
    written this step.
    Attention of a sequence at position p reads p + 1 cached rows; the pool
    reads the first block's rows 0..p, or with running sums (steady state)
    the previous row, the new row and the kept fp32 sums, or nothing of its
    own when the router block's attention sums those rows as it reads them
    (pool_fused: decode steps without skipped-KV masking or running sums)."""
    L = cfg["n_layers"]
    s = _s(cfg["dtype"])
    row = 2 * cfg["n_kv_heads"] * cfg["head_dim"] * s          # one K row + one V row
    S = int(cfg.get("start_layer", 1))
    used = set(range(S)) | {L - 1}
    kv = 0
    for m, p in zip(masks, positions):
        n_exec = S + 1 + sum(int(v) for v in m)
        kv += n_exec * row * (p + 1)
        used.update(l + S for l, v in enumerate(m) if v)
    weights = len(used) * layer_weight_bytes(cfg)
    if running_pool:
        sums = 2 * cfg["n_kv_heads"] * cfg["head_dim"] * 4
        pool = len(positions) * (2 * row + 2 * sums)
    elif pool_fused:
        pool = 0
    else:
        pool = sum(row * (p + 1) for p in positions)
    dmw = dm_weight_bytes(cfg)
    writes = len(positions) * L * row
    return dict(weights=weights, kv=kv, pool=pool, dm=dmw, kv_writes=writes,
                total=weights + kv + pool + dmw + writes, layers_used=len(used))


def kernel_bytes(cfg: dict, n: int, pos: int) -> dict:
    """Algorithmic bytes of one launch of each decoder-block kernel over n
    routed rows at position pos: the weight matrix once, the activation rows
    it reads and writes (fp32), the new K/V rows, and for attention the K/V
    rows 0..pos of every routed sequence (with its fp32 queries in and
    outputs out).  'attention' covers the score kernel and the chunk merge
    together: the merge's partials are not algorithmic bytes."""
    d, nq, nkv, hd, f = (cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                         cfg["head_dim"], cfg["d_ffn"])
    s = _s(cfg["dtype"])
    qdim = nq * hd
    return dict(
        qkv=(nq + 2 * nkv) * hd * d * s + n * d * 4 + n * qdim * 4 + n * 2 * nkv * hd * s,
        attention=n * 2 * nkv * hd * (pos + 1) * s + 2 * n * qdim * 4,
        o_proj=d * qdim * s + n * qdim * 4 + 2 * n * d * 4,
        gate_up=2 * f * d * s + n * d * 4 + n * f * 4,
        down=d * f * s + n * f * 4 + 2 * n * d * 4,
    )
