"""Pins of the CPU oracle against facts fixed outside it.

Each test checks the oracle against something other than itself: library
routines (torch, Hugging Face's Llama), brute force on tiny inputs, closed
forms, and the structural invariants the paper states (exact budget, dense
equivalence, identity of skipped blocks, zero-filled skipped KV).
"""
import math
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

from oracle import Oracle, bf16_from_double
from paper_2606_09514_amd import synth

from _hf import (bf16_round_f64, hf_decode_rounded_cache, hf_forward, hf_model,
                 hf_model_exact, hf_routed_masked)

SMALL = dict(n_layers=6, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, d_ffn=96,
             dm_hidden=32, dm_act="gelu", rope_theta=1e4, rms_eps=1e-5)


def make(shape=SMALL, dtype="f32", max_ctx=24, seed=0, omega=0.0):
    cfg = synth.model_config(shape, dtype, max_ctx)
    W = synth.model_weights(cfg, seed, "cpu", omega=omega)
    layers = [{k: synth.storage_numpy(v) for k, v in lw.items()} for lw in W["layers"]]
    dm = {k: (synth.storage_numpy(v) if torch.is_tensor(v) else v) for k, v in W["dm"].items()}
    return cfg, layers, dm, Oracle(cfg, layers, dm)


def empty_cache(cfg, orc):
    shp = (cfg["n_kv_heads"], cfg["max_ctx"], cfg["head_dim"])
    kc = [np.zeros(shp, dtype=orc.sdt) for _ in range(cfg["n_layers"])]
    vc = [np.zeros(shp, dtype=orc.sdt) for _ in range(cfg["n_layers"])]
    return kc, vc


def relerr(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))


# ----------------------------------------------------------- storage rounding

def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),      # fp32 subnormals
        (rng.standard_normal(2000) * 1e37).astype(np.float32),
        np.array([0.0, -0.0, 1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 3.4028235e38,
                  -3.4028235e38, np.inf, -np.inf], dtype=np.float32),
    ])
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([bf16_from_double(float(v)) for v in vals], dtype=np.uint16)
    assert np.array_equal(got, ref)
    assert bf16_from_double(float("nan")) & 0x7F80 == 0x7F80


def test_single_rounding_helper_matches_oracle_on_doubles():
    """The tests' double -> bf16 helper (torch's float32 path with the
    double-rounding case decided by the double) and the oracle's direct
    rounding agree, including doubles just off a bf16 midpoint, where a
    float32 intermediate would round the wrong way."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal(20000) * np.exp2(rng.integers(-20, 20, 20000))
    # bf16 midpoints nudged by less than a float32 ulp either way
    mid = (torch.from_numpy(rng.standard_normal(4000).astype(np.float32)).view(torch.int32)
           & ~0xFFFF | 0x8000).view(torch.float32).to(torch.float64).numpy()
    x = np.concatenate([x, mid, mid * (1 + 2.0 ** -40), mid * (1 - 2.0 ** -40)])
    ref = np.array([bf16_from_double(float(v)) for v in x], dtype=np.uint16)
    got = bf16_round_f64(torch.from_numpy(x)).to(torch.float32).view(torch.int32).numpy()
    assert np.array_equal(((got >> 16) & 0xFFFF).astype(np.uint16), ref)


# --------------------------------------------------------- bf16 KV storage
#
# In bf16 mode a block stores the new K row after the rotary embedding and
# the new V row, each rounded once to bf16, and attention reads the stored
# (rounded) rows back, the new row included (App. "Background", KV-cache
# equation; Sec. 5 runs the model in bf16).  Pinned against Hugging Face's
# projections and rotary embedding in float64.

def _bf16_bits(a):
    bits = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).to(
        torch.float32).view(torch.int32).numpy()
    return ((bits >> 16) & 0xFFFF).astype(np.uint16)


@pytest.mark.parametrize("pos", [0, 5])
def test_bf16_new_kv_row_is_rounded_rotated_projection(pos):
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    cfg, layers, dm, orc = make(dtype="bf16")
    nq, nkv, hd, d = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"], cfg["d_model"]
    rng = np.random.default_rng(21)
    kc, vc = empty_cache(cfg, orc)
    shp = (nkv, pos, hd)
    to_bf = lambda a: torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).view(
        torch.int16).numpy().view(np.uint16)
    kc[1][:, :pos], vc[1][:, :pos] = to_bf(rng.standard_normal(shp)), to_bf(rng.standard_normal(shp))
    before_k, before_v = kc[1].copy(), vc[1].copy()
    h = rng.standard_normal(d) * 2.0
    orc.block(1, kc[1], vc[1], pos, h)

    f64 = lambda a: torch.from_numpy((a.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    w = layers[1]
    u = torch.nn.functional.rms_norm(torch.from_numpy(h)[None], (d,), f64(w["attn_norm"]),
                                     eps=cfg["rms_eps"])
    wqkv = f64(w["wqkv"])
    k = torch.nn.functional.linear(u, wqkv[nq * hd:(nq + nkv) * hd]).view(1, nkv, 1, hd)
    v = torch.nn.functional.linear(u, wqkv[(nq + nkv) * hd:]).view(nkv, hd)
    inv = 1.0 / (cfg["rope_theta"] ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    emb = torch.cat([pos * inv, pos * inv])[None, None]
    _, k_rot = apply_rotary_pos_emb(k, k, emb.cos(), emb.sin())
    k_rot = k_rot.view(nkv, hd)
    assert np.array_equal(kc[1][:, pos], _bf16_bits(bf16_round_f64(k_rot).numpy()))
    assert np.array_equal(vc[1][:, pos], _bf16_bits(bf16_round_f64(v).numpy()))
    if pos > 0:
        # rotating after rounding would store other bits for most entries
        assert not np.array_equal(kc[1][:, pos], _bf16_bits(
            apply_rotary_pos_emb(bf16_round_f64(k), k, emb.cos(), emb.sin())[0].view(nkv, hd)))
    # no other row is touched
    mask = np.ones(cfg["max_ctx"], dtype=bool)
    mask[pos] = False
    assert np.array_equal(kc[1][:, mask], before_k[:, mask])
    assert np.array_equal(vc[1][:, mask], before_v[:, mask])


def test_bf16_first_row_attention_returns_the_rounded_v():
    """With one cached row (position 0) the softmax weight is 1, so each
    query head's attention output is its KV group's stored V row: the
    block's output equals Hugging Face's block fed the bf16-rounded V.  The
    unrounded V is ~1e-3 relative away (bf16 has 8 significant bits), far
    outside the tolerance."""
    cfg, layers, dm, orc = make(dtype="bf16")
    d = cfg["d_model"]
    hf = hf_model_exact(cfg, layers, [1])
    x = synth.hidden_inputs(1, d, seed=22).numpy().astype(np.float64) * 3.0
    kc, vc = empty_cache(cfg, orc)
    got = orc.block(1, kc[1], vc[1], 0, x[0])
    ref_r, _ = hf_decode_rounded_cache(hf, x)
    ref_u, _ = hf_decode_rounded_cache(hf, x, round_kv=lambda t: t)
    assert relerr(got, ref_r[0]) < 1e-12, relerr(got, ref_r[0])
    assert relerr(got, ref_u[0]) > 1e-6


def _f32_round(t):
    return t.to(torch.float32).to(torch.float64)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("route", [None, (1, 0, 1, 1)])
def test_decode_equals_hf_with_storage_rounded_cache(dtype, route):
    """A sequence (every routable block, or a fixed route, i.e. the dense
    sub-model) against Hugging Face's float64 token-by-token decode whose
    cache stores each new K/V row rounded to the storage dtype after the
    rotary embedding: hidden states to 1e-10 and every stored cache row bit
    for bit.  In bf16, rounding before the rotary embedding, or attending to
    the unrounded new row, moves the hidden states by ~1e-6."""
    cfg, layers, dm, orc = make(dtype=dtype)
    rnd = bf16_round_f64 if dtype == "bf16" else _f32_round
    bits = _bf16_bits if dtype == "bf16" else (lambda a: a.astype(np.float32))
    L, T = cfg["n_layers"], 10
    keep = list(range(L)) if route is None else [0] + [1 + i for i, r in enumerate(route) if r] + [L - 1]
    xs = synth.hidden_inputs(T, cfg["d_model"], seed=23).numpy()
    r = None if route is None else np.array(route, dtype=np.uint8)
    got, execs, _, (kc, vc) = run_sequence(cfg, orc, xs, k=orc.L_mid if r is None else int(r.sum()),
                                           route=r)
    ref, kv = hf_decode_rounded_cache(hf_model_exact(cfg, layers, keep), xs, round_kv=rnd)
    assert relerr(got, ref) < 1e-10, relerr(got, ref)
    for j, li in enumerate(keep):
        assert np.array_equal(kc[li][:, :T], bits(kv[j][0]))
        assert np.array_equal(vc[li][:, :T], bits(kv[j][1]))
    # the same sequence with an unrounded cache differs by far more
    ref_u, _ = hf_decode_rounded_cache(hf_model_exact(cfg, layers, keep), xs,
                                       round_kv=lambda t: t)
    assert relerr(ref_u, ref) > (1e-7 if dtype == "bf16" else 1e-14)


# ------------------------------------------------------------ block pieces

def test_rmsnorm_matches_torch_and_closed_form():
    cfg, layers, dm, orc = make()
    rng = np.random.default_rng(2)
    h = rng.standard_normal(cfg["d_model"]) * 3.0
    g = layers[0]["attn_norm"]
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h)[None], (cfg["d_model"],),
                                       torch.from_numpy(g.astype(np.float64)),
                                       eps=cfg["rms_eps"])[0].numpy()
    assert relerr(orc.rmsnorm(h, g), ref) < 1e-13
    # constant input c: every output is c / sqrt(c^2 + eps) * g
    c = 0.37
    one = np.ones(cfg["d_model"], dtype=np.float32)
    out = orc.rmsnorm(np.full(cfg["d_model"], c), one)
    assert np.allclose(out, c / math.sqrt(c * c + cfg["rms_eps"]), rtol=0, atol=1e-15)


def test_rope_pins():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    cfg, _, _, orc = make()
    hd = cfg["head_dim"]
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal(hd), rng.standard_normal(hd)
    # identity at position 0, norm preserved everywhere
    assert np.array_equal(orc.rope(q, 0), q)
    for p in (1, 7, 300, 8191):
        assert abs(np.linalg.norm(orc.rope(q, p)) - np.linalg.norm(q)) < 1e-12
    # relative position: <R_m q, R_n k> depends only on m - n
    a = orc.rope(q, 9) @ orc.rope(k, 4)
    b = orc.rope(q, 105) @ orc.rope(k, 100)
    assert abs(a - b) < 1e-12
    # the library rotary embedding (angles in fp32 there, hence the tolerance)
    inv = 1.0 / (cfg["rope_theta"] ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    for p in (1, 5, 17):
        ang = p * inv
        emb = torch.cat([ang, ang])
        qe, _ = apply_rotary_pos_emb(torch.from_numpy(q)[None, None, None],
                                     torch.from_numpy(k)[None, None, None],
                                     emb.cos()[None], emb.sin()[None])
        assert np.max(np.abs(qe[0, 0, 0].numpy() - orc.rope(q, p))) < 1e-12


# ------------------------------------------------- dense equivalence and routes

def run_sequence(cfg, orc, xs, k, route=None):
    kc, vc = empty_cache(cfg, orc)
    outs, execs, masks = [], [], []
    for t, x in enumerate(xs):
        h, mask, _, _, n_exec = orc.decode_seq(kc, vc, t, k, x, route=route)
        outs.append(h)
        execs.append(n_exec)
        masks.append(mask)
    return np.array(outs), execs, masks, (kc, vc)


def test_all_layers_equals_dense_forward():
    """k = L_mid: the routed decode is the dense causal forward (Eq. 1, M = 1)."""
    cfg, layers, dm, orc = make()
    xs = synth.hidden_inputs(12, cfg["d_model"], seed=5).numpy()
    got, execs, _, _ = run_sequence(cfg, orc, xs, k=orc.L_mid)
    ref = hf_forward(hf_model(cfg, layers, list(range(cfg["n_layers"]))), xs)
    assert relerr(got, ref) < 1e-5, relerr(got, ref)
    assert all(e == cfg["n_layers"] for e in execs)


def test_k0_equals_first_and_last_block_model():
    cfg, layers, dm, orc = make()
    xs = synth.hidden_inputs(9, cfg["d_model"], seed=6).numpy()
    got, execs, masks, _ = run_sequence(cfg, orc, xs, k=0)
    ref = hf_forward(hf_model(cfg, layers, [0, cfg["n_layers"] - 1]), xs)
    assert relerr(got, ref) < 1e-5
    assert all(e == 2 for e in execs) and all(m.sum() == 0 for m in masks)


def test_constant_route_equals_sub_model():
    """Skipped blocks are never read under a fixed route: the result is the
    dense forward of {first} + S + {last}."""
    cfg, layers, dm, orc = make()
    route = np.array([0, 1, 0, 1], dtype=np.uint8)       # routable layers 2 and 4
    xs = synth.hidden_inputs(10, cfg["d_model"], seed=7).numpy()
    got, execs, _, _ = run_sequence(cfg, orc, xs, k=2, route=route)
    ref = hf_forward(hf_model(cfg, layers, [0, 2, 4, 5]), xs)
    assert relerr(got, ref) < 1e-5
    assert all(e == 4 for e in execs)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_exact_budget_every_k(dtype):
    """Every sequence executes exactly k + 2 blocks and selects k layers."""
    cfg, layers, dm, orc = make(dtype=dtype, omega=0.1)
    xs = synth.hidden_inputs(6, cfg["d_model"], seed=8).numpy()
    for k in range(orc.L_mid + 1):
        _, execs, masks, _ = run_sequence(cfg, orc, xs, k=k)
        assert all(e == k + 2 for e in execs)
        assert all(int(m.sum()) == k for m in masks)


def test_routes_deterministic_under_seed():
    outs = []
    for _ in range(2):
        cfg, layers, dm, orc = make(omega=0.1, seed=11)
        xs = synth.hidden_inputs(8, cfg["d_model"], seed=12).numpy()
        h, _, masks, _ = run_sequence(cfg, orc, xs, k=2)
        outs.append((h.tobytes(), np.array(masks).tobytes()))
    assert outs[0] == outs[1]


def test_thread_count_does_not_change_results():
    code = ("import sys; sys.path.insert(0, %r); sys.path.insert(0, %r)\n"
            "import hashlib, numpy as np\n"
            "from test_oracle_pins import make, run_sequence\n"
            "from paper_2606_09514_amd import synth\n"
            "cfg, l, d, o = make(shape=dict(n_layers=4, d_model=256, n_heads=4, n_kv_heads=2,"
            " head_dim=64, d_ffn=512, dm_hidden=64, dm_act='silu', rope_theta=1e4,"
            " rms_eps=1e-5), omega=0.1)\n"
            "xs = synth.hidden_inputs(4, 256, seed=1).numpy()\n"
            "h, _, m, _ = run_sequence(cfg, o, xs, k=1)\n"
            "print(hashlib.sha256(h.tobytes() + np.array(m).tobytes()).hexdigest())\n"
            % (os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
               os.path.dirname(os.path.abspath(__file__))))
    digests = []
    for n in ("1", "4"):
        env = dict(os.environ, OMP_NUM_THREADS=n)
        r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True,
                           text=True, check=True)
        digests.append(r.stdout.strip().splitlines()[-1])
    assert digests[0] == digests[1]


# -------------------------------------------------------------------- router

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pool_brute_force(dtype):
    cfg, layers, dm, orc = make(dtype=dtype)
    rng = np.random.default_rng(4)
    shp = (cfg["n_kv_heads"], cfg["max_ctx"], cfg["head_dim"])
    if dtype == "bf16":
        mk = lambda: torch.from_numpy(rng.standard_normal(shp).astype(np.float32)).to(
            torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        up = lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    else:
        mk = lambda: rng.standard_normal(shp).astype(np.float32)
        up = lambda a: a.astype(np.float64)
    kc, vc = mk(), mk()
    for pos in (0, 1, 2):
        z = orc.pool(kc, vc, pos)
        n = cfg["n_kv_heads"] * cfg["head_dim"]
        for g in range(cfg["n_kv_heads"]):
            for i in range(cfg["head_dim"]):
                sk = sum(up(kc[g, j, i]) for j in range(pos + 1)) / (pos + 1)
                sv = sum(up(vc[g, j, i]) for j in range(pos + 1)) / (pos + 1)
                assert z[g * cfg["head_dim"] + i] == pytest.approx(sk, rel=1e-15, abs=1e-300)
                assert z[n + g * cfg["head_dim"] + i] == pytest.approx(sv, rel=1e-15, abs=1e-300)
    # constant rows pool to that constant
    kc[...] = kc[0, 0, 0]
    vc[...] = vc[1, 0, 3]
    z = orc.pool(kc, vc, 15)
    assert np.all(z[:n] == up(kc[0, 0, 0])) and np.all(z[n:] == up(vc[1, 0, 3]))


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_dm_scores_match_torch(act):
    shape = dict(SMALL, dm_act=act)
    cfg, layers, dm, orc = make(shape=shape, omega=0.1)
    din = 2 * cfg["n_kv_heads"] * cfg["head_dim"] + cfg["d_model"]
    z = np.random.default_rng(9).standard_normal(din)
    T = lambda a: torch.from_numpy(a.astype(np.float64))
    a = torch.nn.functional.linear(T(z), T(dm["w1"]), T(dm["b1"]))
    a = torch.nn.functional.gelu(a) if act == "gelu" else torch.nn.functional.silu(a)
    s = torch.nn.functional.linear(a, T(dm["w2"]), T(dm["b2"])) + 0.1 * T(dm["prior"])
    got = orc.dm_scores(z)
    assert np.array_equal(got, s.numpy().astype(np.float32)) or \
        np.max(np.abs(got - s.numpy())) < 1e-7


def test_dm_constant_scores_select_lowest_indices():
    cfg, layers, dm, _ = make()
    dm2 = dict(dm, w2=np.zeros_like(dm["w2"]), b2=np.full_like(dm["b2"], 0.25), prior=None)
    orc = Oracle(cfg, layers, dm2)
    kc, vc = empty_cache(cfg, orc)
    for k in range(orc.L_mid + 1):
        _, mask, scores, margin, _ = orc.decode_seq(kc, vc, 0, k, np.ones(cfg["d_model"]))
        assert np.all(scores == np.float32(0.25))
        assert list(mask) == [1] * k + [0] * (orc.L_mid - k)
        assert margin == (math.inf if k in (0, orc.L_mid) else 0.0)


@pytest.mark.parametrize("ctx", ["kv", "k", "v", "k+v"])
def test_router_context_variants_brute_force(ctx):
    """Sec. 4.3 features G_t in {K, V, K + V} (and the [K | V] default of
    this implementation): head-major means of the stored first-layer rows
    over 0..pos, computed here by a plain numpy mean, followed by h; the
    Decision Module takes that many inputs."""
    shape = dict(SMALL, router_ctx=ctx)
    cfg, layers, dm, orc = make(shape=shape, dtype="bf16")
    n = cfg["n_kv_heads"] * cfg["head_dim"]
    assert dm["w1"].shape[1] == synth.context_dim(cfg) == (2 * n if ctx == "kv" else n) + cfg["d_model"]
    rng = np.random.default_rng(9)
    shp = (cfg["n_kv_heads"], cfg["max_ctx"], cfg["head_dim"])
    mk = lambda: torch.from_numpy(rng.standard_normal(shp).astype(np.float32)).to(
        torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    up = lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    kc, vc = mk(), mk()
    h = rng.standard_normal(cfg["d_model"])
    for pos in (0, 3, 11):
        mk_ = up(kc[:, :pos + 1]).mean(axis=1).reshape(-1)      # head-major [n_kv * hd]
        mv_ = up(vc[:, :pos + 1]).mean(axis=1).reshape(-1)
        feat = {"kv": np.concatenate([mk_, mv_]), "k": mk_, "v": mv_, "k+v": mk_ + mv_}[ctx]
        ref = np.concatenate([feat, h])
        z = orc.context(kc, vc, pos, h)
        assert z.shape == ref.shape
        assert np.allclose(z, ref, rtol=1e-14, atol=1e-14)
    # the scores use the variant's context: a different variant gives others
    s = orc.dm_scores(orc.context(kc, vc, 11, h))
    assert s.shape == (orc.L_mid,) and np.all(np.isfinite(s))


def test_omega_zero_ignores_prior():
    cfg, layers, dm, _ = make(omega=0.1)
    z = np.random.default_rng(10).standard_normal(2 * 2 * 16 + 64)
    with_prior_w0 = Oracle(cfg, layers, dict(dm, omega=0.0)).dm_scores(z)
    without = Oracle(cfg, layers, dict(dm, prior=None)).dm_scores(z)
    assert np.array_equal(with_prior_w0, without)


def test_topk_matches_stable_sort():
    rng = np.random.default_rng(11)
    for trial in range(300):
        n = int(rng.integers(1, 40))
        s = rng.integers(-3, 4, size=n).astype(np.float32) * 0.5   # many ties
        if trial % 5 == 0:
            s[rng.integers(0, n)] = np.nan
        if trial % 7 == 0:
            s[rng.integers(0, n)] = -0.0
        k = int(rng.integers(0, n + 1))
        key = lambda i: (1, 0.0, i) if np.isnan(s[i]) else (0, -float(s[i]), i)
        order = sorted(range(n), key=key)
        mask, margin = Oracle.topk(s, k)
        assert sorted(np.nonzero(mask)[0].tolist()) == sorted(order[:k])
        if 0 < k < n:
            m = float(s[order[k - 1]]) - float(s[order[k]])
            assert margin == (0.0 if math.isnan(m) else m)
        else:
            assert margin == math.inf
    with pytest.raises(ValueError):
        Oracle.topk(np.zeros(3, np.float32), 4)


# --------------------------------------------------------- skipped-layer KV

def test_skipped_layer_kv_is_zero_and_attended_as_zero():
    """Sec. 6: skipped layers keep zero-filled K/V, which later steps attend
    as ordinary entries.  Built so the routable block adds exactly the mean
    of its V cache over positions 0..pos (W_q = 0 gives uniform attention,
    W_o = I, no MLP); the outer blocks are identities (W_o = W_down = 0)."""
    shape = dict(n_layers=3, d_model=4, n_heads=1, n_kv_heads=1, head_dim=4, d_ffn=4,
                 dm_hidden=4, dm_act="silu", rope_theta=1e4, rms_eps=1e-5)
    cfg, layers, dm, _ = make(shape=shape, max_ctx=4)
    for lw in layers:
        lw["wo"][...] = 0
        lw["wdown"][...] = 0
    layers[1]["wqkv"][:4] = 0                      # q rows
    layers[1]["wo"][...] = np.eye(4, dtype=np.float32)
    orc = Oracle(cfg, layers, dm)
    kc, vc = empty_cache(cfg, orc)
    for a in kc + vc:            # stale contents: every slot read must be written first
        a[...] = 7.0
    rng = np.random.default_rng(12)
    x0, x1 = rng.standard_normal(4).astype(np.float32), rng.standard_normal(4).astype(np.float32)
    h0, *_ = orc.decode_seq(kc, vc, 0, 0, x0, route=np.array([0], np.uint8))
    assert np.array_equal(h0, x0.astype(np.float64))          # blocks 0 and 2 are identities
    assert np.all(kc[1][:, 0] == 0) and np.all(vc[1][:, 0] == 0)
    assert np.any(kc[0][:, 0] != 0)
    h1, *_ = orc.decode_seq(kc, vc, 1, 1, x1, route=np.array([1], np.uint8))
    v1 = vc[1][0, 1].astype(np.float64)
    assert np.any(v1 != 0)
    # literal zero-fill: the skipped slot counts in the softmax with value 0
    assert np.allclose(h1, x1 + (0.0 + v1) / 2.0, rtol=0, atol=1e-14)


# --------------------------------------------------- skipped-KV masking

def test_masked_skipped_kv_leaves_the_slot_out():
    """Masking variant of the skipped-layer KV (the alternative to zero-fill
    that the paper's conclusion names as future work): the hand case of the
    zero-fill test, where the routable block adds the mean of its V rows over
    the positions it attends; with the slot of the skipped step left out it
    adds exactly the new row's V."""
    shape = dict(n_layers=3, d_model=4, n_heads=1, n_kv_heads=1, head_dim=4, d_ffn=4,
                 dm_hidden=4, dm_act="silu", rope_theta=1e4, rms_eps=1e-5)
    cfg, layers, dm, _ = make(shape=shape, max_ctx=4)
    for lw in layers:
        lw["wo"][...] = 0
        lw["wdown"][...] = 0
    layers[1]["wqkv"][:4] = 0
    layers[1]["wo"][...] = np.eye(4, dtype=np.float32)
    orc = Oracle(cfg, layers, dm)
    kc, vc = empty_cache(cfg, orc)
    execs = [np.full(cfg["max_ctx"], 9, np.uint8) for _ in range(3)]   # stale contents
    rng = np.random.default_rng(12)
    x0, x1 = rng.standard_normal(4).astype(np.float32), rng.standard_normal(4).astype(np.float32)
    orc.decode_seq(kc, vc, 0, 0, x0, route=np.array([0], np.uint8), execs=execs)
    assert [e[0] for e in execs] == [1, 0, 1]
    assert np.all(kc[1][:, 0] == 0) and np.all(vc[1][:, 0] == 0)   # still zero-filled
    h1, *_ = orc.decode_seq(kc, vc, 1, 1, x1, route=np.array([1], np.uint8), execs=execs)
    assert [e[1] for e in execs] == [1, 1, 1]
    v1 = vc[1][0, 1].astype(np.float64)
    assert np.allclose(h1, x1 + v1, rtol=0, atol=1e-14)


def test_masked_routes_equal_per_block_subsequence_forward():
    """Random per-token routes with masking equal an independent cache-free
    forward (Hugging Face blocks, float64) in which each block runs causally
    over the tokens that execute it, at their original positions."""
    cfg, layers, dm, orc = make()
    T, L = 14, cfg["n_layers"]
    rng = np.random.default_rng(31)
    routes = (rng.random((T, orc.L_mid)) < 0.5).astype(np.uint8)
    xs = synth.hidden_inputs(T, cfg["d_model"], seed=32).numpy()
    kc, vc = empty_cache(cfg, orc)
    execs = [np.zeros(cfg["max_ctx"], np.uint8) for _ in range(L)]
    got = np.array([orc.decode_seq(kc, vc, t, int(routes[t].sum()), xs[t], route=routes[t],
                                   execs=execs)[0] for t in range(T)])
    ref = hf_routed_masked(hf_model(cfg, layers, list(range(L))), xs, routes)
    assert relerr(got, ref) < 1e-5, relerr(got, ref)
    # and it is not the zero-fill result
    kc2, vc2 = empty_cache(cfg, orc)
    zf = np.array([orc.decode_seq(kc2, vc2, t, int(routes[t].sum()), xs[t], route=routes[t])[0]
                   for t in range(T)])
    assert relerr(zf, ref) > 1e-3


# -------------------------------------------- prior normalisation (App. B)

def test_prior_normalize_hand_case():
    """Four Taylor scores 1..4: log(1 + x) and the robust z keep the order, so
    u = (1 + rank) / 5 = 0.2 .. 0.8, and Eq. 2 standardises it: mean 0.5,
    population std sqrt(0.05)."""
    from oracle import prior_normalize
    got = prior_normalize([1.0, 2.0, 3.0, 4.0], 1)
    u = np.array([0.2, 0.4, 0.6, 0.8])
    assert np.allclose(got, (u - 0.5) / (np.sqrt(0.05) + 1e-6), rtol=0, atol=1e-12)


@pytest.mark.parametrize("kind", [0, 1, 2])
def test_prior_normalize_depends_only_on_order(kind):
    """Without winsorising, steps (ii) and (iii) are increasing maps, so u is
    the rank transform of the direction-unified indicator: scipy's average
    ranks give the same prior (ties from clipping at 0 included)."""
    from scipy.stats import rankdata
    from oracle import prior_normalize
    rng = np.random.default_rng(40 + kind)
    raw = rng.standard_normal(30) * 3.0
    raw[[4, 9]] = -1.0                      # clipped to 0 together (kinds 0 and 1)
    raw[[11, 20]] = raw[5]                  # exact ties
    x = 1.0 - raw if kind == 2 else np.maximum(raw, 0.0)
    u = rankdata(x, method="average") / (raw.size + 1)      # 1-based ranks: 1 + rank0
    ref = (u - u.mean()) / (u.std() + 1e-6)
    assert np.allclose(prior_normalize(raw, kind), ref, rtol=0, atol=1e-12)
    # cosine: a more similar block (smaller change) is less important
    if kind == 2:
        p = prior_normalize([0.9, 0.5, 0.1], 2)
        assert p[0] < p[1] < p[2]


def test_prior_normalize_winsor_ties():
    """Winsorising clips the robust z-scores: values beyond the clip share the
    clipped value and therefore one mean rank (numpy percentile and scipy
    ranks as the reference for this special case)."""
    from scipy.stats import rankdata
    from oracle import prior_normalize
    raw = np.array([0.0, 0.1, 0.2, 0.3, 0.4, 50.0, 80.0, 200.0])
    x = np.log1p(raw)
    q25, q50, q75 = np.percentile(x, [25, 50, 75])
    z = np.clip((x - q50) / (q75 - q25 + 1e-6), -1.0, 1.0)
    assert np.sum(z == 1.0) >= 2
    u = rankdata(z, method="average") / (raw.size + 1)
    ref = (u - u.mean()) / (u.std() + 1e-6)
    assert np.allclose(prior_normalize(raw, 1, winsor=1.0), ref, rtol=0, atol=1e-12)


# --------------------------------------------------- Budget Predictor

def _predictor(cfg, hidden=16, seed=3):
    return {k: synth.storage_numpy(v) for k, v in synth.predictor_weights(cfg, hidden, seed).items()}


def test_predictor_argmax_and_ties():
    """Sec. 4.4: k_hat = argmax over k in {1..L-2}; with W2 = 0 the logits are
    b2, so a one-hot b2 picks its action, equal logits pick the smaller k and
    a NaN logit never wins."""
    cfg, layers, dm, orc = make()
    pred = _predictor(cfg)
    pred["w2"][...] = 0
    z = np.random.default_rng(1).standard_normal(synth.context_dim(cfg))
    for j in range(orc.L_mid):
        pred["b2"][...] = 0
        pred["b2"][j] = 0.5
        orc.set_predictor(pred)
        k, lg, margin = orc.predict_budget(z)
        assert k == j + 1 and margin == pytest.approx(0.5)
    pred["b2"][...] = 0.25
    orc.set_predictor(pred)
    assert orc.predict_budget(z)[0] == 1
    pred["b2"][0] = np.nan
    pred["b2"][2] = 0.5
    orc.set_predictor(pred)
    assert orc.predict_budget(z)[0] == 3


@pytest.mark.parametrize("act", ["silu", "gelu"])
def test_predictor_mlp_matches_torch(act):
    """The head's two linear layers and activation reduce to torch's linear
    and SiLU / exact GELU (float64), rounded to fp32."""
    shape = dict(SMALL, dm_act=act)
    cfg, layers, dm, orc = make(shape=shape)
    pred = _predictor(cfg, hidden=24, seed=5)
    orc.set_predictor(pred)
    z = np.random.default_rng(2).standard_normal(synth.context_dim(cfg))
    t = {k: torch.from_numpy(v.astype(np.float64)) for k, v in pred.items()}
    a = torch.nn.functional.linear(torch.from_numpy(z), t["w1"], t["b1"])
    a = torch.nn.functional.silu(a) if act == "silu" else torch.nn.functional.gelu(a)
    ref = torch.nn.functional.linear(a, t["w2"], t["b2"]).numpy()
    k, lg, _ = orc.predict_budget(z)
    assert np.allclose(lg, ref.astype(np.float32), rtol=1e-6, atol=1e-7)
    assert k == int(np.argmax(ref.astype(np.float32))) + 1


def test_auto_budget_step_equals_budgeted_step():
    """Without a budget the step runs exactly k_hat + 2 blocks, as the
    budgeted step with k = k_hat does, and b_hat = (k_hat + 2) / L maps back
    to k_hat through the Eq. 2 rounding."""
    from paper_2606_09514_amd import costmodel
    cfg, layers, dm, orc = make(omega=0.1)
    orc.set_predictor(_predictor(cfg, hidden=32, seed=7))
    xs = synth.hidden_inputs(6, cfg["d_model"], seed=11).numpy()
    kc, vc = empty_cache(cfg, orc)
    kc2, vc2 = empty_cache(cfg, orc)
    seen = set()
    for t, x in enumerate(xs):
        h, k, lg, pm, mask, sc, margin, n_exec = orc.decode_seq_auto(kc, vc, t, x)
        h2, m2, s2, _, n2 = orc.decode_seq(kc2, vc2, t, k, x)
        assert 1 <= k <= orc.L_mid and n_exec == k + 2 and int(mask.sum()) == k
        assert np.array_equal(h, h2) and np.array_equal(mask, m2) and np.array_equal(sc, s2)
        b_hat = (k + 2) / cfg["n_layers"]
        assert costmodel.budget_to_k(b_hat, cfg["n_layers"]) == k
        seen.add(k)


# ------------------------------------------------------------ routed prefill

def prefill(cfg, orc, xs, k, route=None, execs=None):
    kc, vc = empty_cache(cfg, orc)
    h, mask, sc, margin = orc.prefill_seq(kc, vc, xs, k, route=route, execs=execs)
    return h, mask, sc, (kc, vc)


def test_prefill_all_blocks_equals_dense_forward():
    """k = L - 2: the prefill of every prompt token is the dense causal
    forward (Eq. 1 with M = 1)."""
    cfg, layers, dm, orc = make()
    xs = synth.hidden_inputs(11, cfg["d_model"], seed=51).numpy()
    h, mask, _, _ = prefill(cfg, orc, xs, orc.L_mid)
    ref = hf_forward(hf_model(cfg, layers, list(range(cfg["n_layers"]))), xs)
    assert relerr(h, ref) < 1e-5 and mask.sum() == orc.L_mid


def test_prefill_route_and_sub_model():
    """The prompt's route is the planner's decision at the last token: the
    first-layer cache pooled over the prompt and the last token's hidden
    state after the first block (here from a one-block Hugging Face forward);
    every token's output is the dense forward of {first} + S + {last}, and
    the skipped blocks hold zeros over the prompt."""
    cfg, layers, dm, orc = make(omega=0.1)
    n, k, L = 13, 2, cfg["n_layers"]
    xs = synth.hidden_inputs(n, cfg["d_model"], seed=52).numpy()
    h, mask, sc, (kc, vc) = prefill(cfg, orc, xs, k)
    h0 = hf_forward(hf_model(cfg, layers, [0]), xs)[-1]
    s_ref = orc.dm_scores(orc.context(kc[0], vc[0], n - 1, h0))
    assert np.allclose(sc, s_ref, rtol=1e-6, atol=1e-7)
    assert np.array_equal(mask, Oracle.topk(s_ref, k)[0])
    keep = [0] + [l for l in range(1, L - 1) if mask[l - 1]] + [L - 1]
    assert relerr(h, hf_forward(hf_model(cfg, layers, keep), xs)) < 1e-5
    for l in range(1, L - 1):
        if not mask[l - 1]:
            assert np.all(kc[l][:, :n] == 0) and np.all(vc[l][:, :n] == 0)


@pytest.mark.parametrize("masked", [False, True])
def test_prefill_then_decode_equals_token_by_token(masked):
    """Prefill then decode under the prompt's route is, bit for bit, the
    decode of every token one by one under that route (the same arithmetic
    in the same order; caches and, with masking, execution maps equal)."""
    cfg, layers, dm, orc = make(dtype="bf16", omega=0.1)
    n, L = 9, cfg["n_layers"]
    xs = synth.hidden_inputs(n + 3, cfg["d_model"], seed=53).numpy()
    ex1 = [np.zeros(cfg["max_ctx"], np.uint8) for _ in range(L)] if masked else None
    ex2 = [np.zeros(cfg["max_ctx"], np.uint8) for _ in range(L)] if masked else None
    h, mask, _, (kc, vc) = prefill(cfg, orc, xs[:n], 2, execs=ex1)
    kc2, vc2 = empty_cache(cfg, orc)
    for t in range(n):
        h2, *_ = orc.decode_seq(kc2, vc2, t, 2, xs[t], route=mask, execs=ex2)
        assert np.array_equal(h[t], h2)
    for t in range(n, n + 3):
        a, *_ = orc.decode_seq(kc, vc, t, 2, xs[t], route=mask, execs=ex1)
        b, *_ = orc.decode_seq(kc2, vc2, t, 2, xs[t], route=mask, execs=ex2)
        assert np.array_equal(a, b)
    for l in range(L):
        assert np.array_equal(kc[l], kc2[l]) and np.array_equal(vc[l], vc2[l])
        if masked:
            assert np.array_equal(ex1[l], ex2[l])



# ------------------------------------------ start layer of the router (Sec. 4.3)

def _up(a):
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("S", [2, 3])
def test_start_layer_router_context_and_budget(S, dtype):
    """Start layer S: the router reads block S-1's cache (numpy means of its
    stored rows 0..pos) and the hidden state after block S-1 (a Hugging
    Face forward of blocks 0..S-1, which always run); the budget counts the
    blocks S..L-2, so S + 1 + k blocks execute."""
    shape = dict(SMALL, start_layer=S)
    cfg, layers, dm, orc = make(shape=shape, dtype=dtype, omega=0.1)
    L, n = cfg["n_layers"], 8
    assert orc.L_mid == L - 1 - S and dm["w2"].shape[0] == L - 1 - S
    xs = synth.hidden_inputs(n, cfg["d_model"], seed=60 + S).numpy()
    hS = hf_forward(hf_model(cfg, layers, list(range(S))), xs)
    kc, vc = empty_cache(cfg, orc)
    for t in range(n):
        k = t % (orc.L_mid + 1)
        _, mask, sc, _, n_exec = orc.decode_seq(kc, vc, t, k, xs[t])
        assert n_exec == S + 1 + k and int(mask.sum()) == k
        z = np.concatenate([_up(kc[S - 1][:, :t + 1]).mean(axis=1).reshape(-1),
                            _up(vc[S - 1][:, :t + 1]).mean(axis=1).reshape(-1), hS[t]])
        s_ref = orc.dm_scores(z)
        tol = 1e-5 if dtype == "f32" else 2e-3
        assert np.max(np.abs(sc - s_ref)) <= tol * max(1.0, float(np.max(np.abs(s_ref)))), t


@pytest.mark.parametrize("S", [2, 3])
def test_start_layer_fixed_route_is_sub_model(S):
    """Under a fixed route over blocks S..L-2 the decode (and the prefill) is
    the dense forward of blocks 0..S-1, the selected ones and L-1; skipped
    blocks hold zeros.  With S = L-1 nothing is routable: the dense model."""
    shape = dict(SMALL, start_layer=S)
    cfg, layers, dm, orc = make(shape=shape)
    L = cfg["n_layers"]
    route = np.zeros(orc.L_mid, np.uint8)
    route[-1] = 1
    keep = list(range(S)) + [S + i for i in range(orc.L_mid) if route[i]] + [L - 1]
    xs = synth.hidden_inputs(10, cfg["d_model"], seed=70 + S).numpy()
    ref = hf_forward(hf_model(cfg, layers, keep), xs)
    got, execs, _, (kc, vc) = run_sequence(cfg, orc, xs, k=1, route=route)
    assert relerr(got, ref) < 1e-5 and all(e == len(keep) for e in execs)
    h, _, _, (pk, pv) = prefill(cfg, orc, xs, 1, route=route)
    assert relerr(h, ref) < 1e-5
    for i in range(orc.L_mid):
        if not route[i]:
            assert np.all(kc[S + i][:, :10] == 0) and np.all(pk[S + i][:, :10] == 0)
    full = dict(SMALL, start_layer=L - 1)
    cfg2, layers2, _, orc2 = make(shape=full)
    assert orc2.L_mid == 0
    got2, execs2, _, _ = run_sequence(cfg2, orc2, xs, k=0)
    assert relerr(got2, hf_forward(hf_model(cfg2, layers2, list(range(L))), xs)) < 1e-5
    assert all(e == L for e in execs2)


def test_start_layer_prefill_route_from_block_s_minus_1():
    """Prefill at start layer 2: the prompt's route comes from block 1's
    cache over the prompt and the last token after blocks 0 and 1."""
    shape = dict(SMALL, start_layer=2)
    cfg, layers, dm, orc = make(shape=shape, omega=0.1)
    n, k, L = 12, 1, cfg["n_layers"]
    xs = synth.hidden_inputs(n, cfg["d_model"], seed=75).numpy()
    h, mask, sc, (kc, vc) = prefill(cfg, orc, xs, k)
    h1 = hf_forward(hf_model(cfg, layers, [0, 1]), xs)[-1]
    s_ref = orc.dm_scores(orc.context(kc[1], vc[1], n - 1, h1))
    assert np.allclose(sc, s_ref, rtol=1e-6, atol=1e-7)
    keep = [0, 1] + [2 + i for i in range(orc.L_mid) if mask[i]] + [L - 1]
    assert relerr(h, hf_forward(hf_model(cfg, layers, keep), xs)) < 1e-5


# ------------------------------------------------- batch-level path grouping

def test_group_by_route_matches_sorted():
    """Path grouping against Python's stable sort on (route, index), with
    routes read as run / skip, and groups as maximal runs of equal routes;
    many duplicate routes, bytes other than 0 and 1, one routable block."""
    from oracle import group_by_route
    rng = np.random.default_rng(31)
    for trial in range(200):
        B = int(rng.integers(1, 70))
        n = int(rng.integers(1, 12)) if trial % 10 else 1
        # few distinct routes so that groups have several members
        pool = rng.integers(0, 2, size=(int(rng.integers(1, 6)), n)).astype(np.uint8)
        m = pool[rng.integers(0, len(pool), size=B)].copy()
        m[m == 1] = rng.choice(np.array([1, 7, 255], np.uint8), size=int((m == 1).sum()))
        perm, starts = group_by_route(m)
        key = lambda b: (tuple(int(v != 0) for v in m[b]), b)
        ref = sorted(range(B), key=key)
        assert perm.tolist() == ref
        routes = [key(b)[0] for b in ref]
        ref_starts = [i for i in range(B) if i == 0 or routes[i] != routes[i - 1]] + [B]
        assert starts.tolist() == ref_starts
    # degenerate cases: every route equal (one group), every route distinct
    perm, starts = group_by_route(np.ones((5, 3), np.uint8))
    assert perm.tolist() == [0, 1, 2, 3, 4] and starts.tolist() == [0, 5]
    m = np.array([[1, 1], [0, 1], [1, 0], [0, 0]], np.uint8)
    perm, starts = group_by_route(m)
    assert perm.tolist() == [3, 1, 2, 0] and starts.tolist() == [0, 1, 2, 3, 4]
