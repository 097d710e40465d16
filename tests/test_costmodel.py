"""Host cost model pinned to the paper's worked example (App. C.2) and its
budget arithmetic (Eq. 2, Sec. 4.4, Sec. 5 settings)."""
import json
import os

import pytest

from paper_2606_09514_amd import costmodel as cm
from paper_2606_09514_amd import synth

G = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "app_c2_worked_example.json")))


def test_app_c2_flop_counts_exact():
    i = G["inputs"]
    assert cm.dm_flops(i["B"], i["T"], i["d"], i["r"], i["L"], i["I"]) == G["F_DM"]
    assert cm.layer_flops(i["T"], i["d"], i["d_c"]) == G["F_layer"]
    assert cm.model_flops(0.875, i["L"], i["T"], i["d"], i["d_c"]) == G["F_model_b0875"]
    assert cm.model_flops(0.5, i["L"], i["T"], i["d"], i["d_c"]) == G["F_model_b05"]


def test_app_c2_overhead_ratio():
    i = G["inputs"]
    for b, key in ((0.875, "rho_b0875"), (0.5, "rho_b05")):
        rho = cm.dm_overhead(b, i["B"], i["T"], i["d"], i["d_c"], i["r"], i["L"], i["I"])
        assert rho == pytest.approx(G[key], rel=5e-3)


def test_budget_to_k_matches_removed_block_counts():
    for rm, b in G["removed_blocks_llama32"].items():
        k = cm.budget_to_k(b, 32)
        assert 32 - (k + 2) == int(rm[2:])
    # Qwen2.5-7B: 28 layers, removing 4/8/12/16 blocks
    for rm in (4, 8, 12, 16):
        assert cm.budget_to_k((28 - rm) / 28, 28) == 28 - rm - 2
    # inverse map of the Budget Predictor, b = (k + 2) / L
    for k in range(31):
        assert cm.budget_to_k(cm.k_to_budget(k, 32), 32) == k
    assert cm.budget_to_k(0.01, 32, clamp=True) == 1
    with pytest.raises(ValueError):
        cm.budget_to_k(0.0, 32)


def test_step_bytes_counts_union_of_routes():
    cfg = synth.model_config("llama3_8b", "bf16", 2176)
    W = cm.layer_weight_bytes(cfg)
    assert W == (4096 * 6144 + 4096 * 4096 + 3 * 4096 * 14336 + 2 * 4096) * 2
    m = [[1] * 15 + [0] * 15]
    r = cm.step_bytes(cfg, m, [2048])
    assert r["layers_used"] == 17 and r["weights"] == 17 * W
    row = 2 * 8 * 128 * 2
    assert r["kv"] == 17 * row * 2049 and r["pool"] == row * 2049
    # two sequences with disjoint routes use every layer once
    r2 = cm.step_bytes(cfg, [[1] * 15 + [0] * 15, [0] * 15 + [1] * 15], [10, 20])
    assert r2["layers_used"] == 32 and r2["weights"] == 32 * W
    # the router block's attention summing the pooled rows: no pool reads
    r3 = cm.step_bytes(cfg, m, [2048], pool_fused=True)
    assert r3["pool"] == 0 and r3["total"] == r["total"] - r["pool"]


def test_kernel_bytes_cover_the_block_weights():
    """The per-kernel algorithmic bytes hold each weight matrix once: their
    weight parts sum to a block's weights without the two norm gains, and
    attention scales with the attended rows."""
    cfg = synth.model_config("llama3_8b", "bf16", 4096)
    kb0 = cm.kernel_bytes(cfg, 0, 0)
    weights = kb0["qkv"] + kb0["o_proj"] + kb0["gate_up"] + kb0["down"]
    assert weights == cm.layer_weight_bytes(cfg) - 2 * cfg["d_model"] * 2
    a1 = cm.kernel_bytes(cfg, 1, 2047)["attention"]
    a2 = cm.kernel_bytes(cfg, 2, 2047)["attention"]
    assert a2 == 2 * a1
    assert a1 == 2 * 8 * 128 * 2048 * 2 + 2 * 4096 * 4
