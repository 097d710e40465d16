#!/usr/bin/env python3
"""Benchmark of the budget-routed decode step on one MI355X.

Workload: a Llama-3-8B-shaped random-init model (32 blocks, d 4096, 32/8
heads, FFN 14336, Decision Module hidden 512, bf16 weights and KV cache),
batch 1 with 2048 cached positions, decoding with budgets k in {15, 22, 30}.
Inputs are synthetic (seeded), resident in HBM before timing.

For each k: W untimed warm-up steps, then K timed steps bracketed by a
device synchronisation on both sides; the hidden state is fed back and the
position advances every step.  The headline `value` is tokens/s at the first
budget (k = 15).  The roofline object covers the dominant kernel (the
RMSNorm + gate/up + SwiGLU GEMV of the first block, which runs every step),
timed live with HIP events around that launch inside the timed region.  The
CPU baseline times the oracle on the host cores on a bounded sample of the
same workload.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0   # MI355X HBM3E peak
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "hbm_traffic_llama3_8b_b1_ctx2048.md")
KERNEL_SOURCES = ["paper_2606_09514_amd/csrc/k_gemv.hip", "paper_2606_09514_amd/csrc/epilogue.h",
                  "paper_2606_09514_amd/csrc/buddy_internal.h"]


def measured_traffic():
    """Bytes per launch of the gate/up GEMV from the committed rocprofv3 PMC
    record, or None when the record is missing or the kernel sources changed
    since the counters were taken."""
    import hashlib
    import re
    try:
        text = open(TRAFFIC_RECORD).read()
    except OSError:
        return None
    m = re.search(r"gate_up_traffic_bytes=(\d+) kernel_sources_sha256=([0-9a-f]{64})", text)
    if not m:
        return None
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return int(m.group(1)) if h.hexdigest() == m.group(2) else None


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def run_budget(model, cfg, w, dk, dv, x0, ks, steps, warmup, hip, kernel_layer, exec_map=None,
               running_pool=False, kernel=None, repeats=1):
    """ks: budgets per sequence, or None for budget-free steps (the attached
    Budget Predictor picks them); exec_map: execution map for skipped-KV
    masking, or None for zero-filled skipped KV; running_pool: the planner
    keeps running sums of the first block's rows (fresh state per budget,
    so the first warm-up step sums the whole cache).  The first timed run of
    `steps` steps gives every figure; repeats - 1 further runs over the same
    positions, after it, give only their tokens/s (run_tokens_per_s, and the
    median over all runs)."""
    import numpy as np
    import torch
    from paper_2606_09514_amd import costmodel
    from paper_2606_09514_amd import lib as blib
    from paper_2606_09514_amd import synth

    B, Lm = w.batch, synth.n_mid(cfg)
    hidden = x0.clone()
    masks = torch.zeros((steps, B, Lm), dtype=torch.uint8, device="cuda")
    k_pred = torch.zeros((steps, B), dtype=torch.int32, device="cuda")
    skip = blib.SKIP_KV_ZERO if exec_map is None else blib.SKIP_KV_MASK
    pool = model.pool_state() if running_pool else None

    def step(pos, t=None):
        mo = None if t is None else masks[t]
        if ks is None:
            model.decode_step_auto(dk, dv, hidden, [pos] * B, k_out=k_pred[t or 0], mask_out=mo,
                                   skip_kv=skip, exec_map=exec_map, pool=pool)
        else:
            model.decode_step(dk, dv, hidden, [pos] * B, ks, mask_out=mo, skip_kv=skip,
                              exec_map=exec_map, pool=pool)

    pos = w.ctx
    for _ in range(warmup):
        step(pos)
        pos += 1
    pos0 = pos
    kernel = blib.KERNEL_GATE_UP if kernel is None else kernel
    starts, stops = hip.create(steps), hip.create(steps)
    model.set_timing_events(kernel, kernel_layer, starts, stops)
    positions = []
    torch.cuda.synchronize()
    # an event between consecutive steps on the launch stream: the first and
    # last bracket the timed region, the others give per-step times
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    # host CPU time of the process over the timed steps (the host-routed
    # launch policy waits for each step's route)
    cpu0 = time.process_time()
    evs[0].record()
    for t in range(steps):
        step(pos, t)
        evs[t + 1].record()
        positions.append([pos] * B)
        pos += 1
    torch.cuda.synchronize()
    cpu_ms = (time.process_time() - cpu0) * 1e3
    model.set_timing_events(kernel, kernel_layer, [], [])
    total_ms = evs[0].elapsed_time(evs[steps])
    step_ms = np.array([evs[t].elapsed_time(evs[t + 1]) for t in range(steps)])
    kern_ms = [hip.elapsed_ms(a, b) for a, b in zip(starts, stops)]
    hip.destroy(starts + stops)
    m = masks.cpu().numpy()
    kk = k_pred.cpu().numpy() if ks is None else np.array([ks] * steps)
    # the router block's attention sums the pooled rows unless masking or
    # running sums take the pool kernel
    fused = exec_map is None and not running_pool
    step_bytes = [costmodel.step_bytes(cfg, m[t], positions[t], running_pool, fused)
                  for t in range(steps)]
    total_bytes = sum(s["total"] for s in step_bytes)
    assert all(int(m[t, b].sum()) == kk[t, b] for t in range(steps) for b in range(B))
    distinct = len({m[t].tobytes() for t in range(steps)})
    # batch-level path grouping of every timed step's executed routes (after
    # the timed region): groups of identical routes, and the block runs that
    # serving each group as its own sub-batch would take (k + 2 blocks per
    # group) against the blocks the per-block compaction runs
    groups, per_path = [], []
    if B > 1:
        perm = torch.empty(B, dtype=torch.int32, device="cuda")
        starts = torch.empty(B + 1, dtype=torch.int32, device="cuda")
        ng = torch.empty(1, dtype=torch.int32, device="cuda")
        for t in range(steps):
            blib.group_by_route(masks[t], perm, starts, ng)
            g = int(ng.item())
            st = starts[:g + 1].cpu().numpy()
            first = perm.cpu().numpy()[st[:-1]]
            groups.append(g)
            per_path.append(int(sum(int(m[t, b].sum()) + 2 for b in first)))
    # further timed runs over the same positions: tokens/s only
    runs = [B * steps / (total_ms / 1e3)]
    for _ in range(repeats - 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for t in range(steps):
            step(pos0 + t, t)
        e1.record()
        torch.cuda.synchronize()
        runs.append(B * steps / (e0.elapsed_time(e1) / 1e3))
    return dict(ks=ks, total_ms=total_ms, ms_per_step=total_ms / steps,
                run_tokens_per_s=runs, median_tokens_per_s=float(np.median(runs)),
                step_ms_p50=float(np.percentile(step_ms, 50)),
                step_ms_p90=float(np.percentile(step_ms, 90)),
                tokens_per_s=B * steps / (total_ms / 1e3),
                host_cpu_ms_per_step=cpu_ms / steps,
                bytes_per_step=total_bytes / steps,
                step_hbm_frac=total_bytes / (total_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
                layers_used=sum(s["layers_used"] for s in step_bytes) / steps,
                distinct_routes=distinct, kernel_ms=sum(kern_ms) / len(kern_ms),
                mean_k=float(kk.mean()), hidden=hidden, end_pos=pos,
                route_groups=float(np.mean(groups)) if groups else None,
                per_path_blocks=float(np.mean(per_path)) if per_path else None)


def run_prefill(model, cfg, w, dk, dv, ks_list, reps, warmup):
    """Routed prefill of a prompt of w.ctx tokens per sequence at each
    budget: prompt tokens per second (the call returns after the device)."""
    import torch
    from paper_2606_09514_amd import synth

    B, n = w.batch, w.ctx
    x = synth.hidden_inputs(B * n, cfg["d_model"], seed=5, device="cuda").reshape(B, n, -1)
    out = {}
    for k in ks_list:
        hidden = torch.empty_like(x)
        times = []
        for r in range(warmup + reps):
            hidden.copy_(x)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            model.prefill(dk, dv, hidden, [n] * B, [k] * B)
            torch.cuda.synchronize()
            if r >= warmup:
                times.append(time.perf_counter() - t0)
        ms = 1e3 * sorted(times)[len(times) // 2]
        out[str(k)] = dict(ms_per_prefill=round(ms, 3), tokens_per_s=round(B * n / (ms / 1e3), 1))
        log(f"prefill k={k}: {ms:.2f} ms for {B} x {n} tokens, {B * n / (ms / 1e3):.0f} tokens/s")
    return out


KERNEL_KINDS = [("qkv", "KERNEL_QKV"), ("attention", "KERNEL_ATTENTION"),
                ("attn_merge", "KERNEL_ATTN_MERGE"), ("o_proj", "KERNEL_O_PROJ"),
                ("gate_up", "KERNEL_GATE_UP"), ("down", "KERNEL_DOWN")]


def per_kernel(model, cfg, w, dk, dv, x0, ks, hip, steps=24, warmup=2):
    """Live launch durations of every kernel of the last block (which runs
    every step and takes the same kernels as a routed block; the first
    block's attention also sums the planner's pool), from the timing hook's
    events on the library's stream, against each kernel's algorithmic bytes
    per launch (attention: the score kernel and the chunk merge together)."""
    from paper_2606_09514_amd import costmodel
    from paper_2606_09514_amd import lib as blib
    us = {}
    last = cfg["n_layers"] - 1
    for name, attr in KERNEL_KINDS:
        r = run_budget(model, cfg, w, dk, dv, x0, ks, steps, warmup, hip, last,
                       kernel=getattr(blib, attr))
        us[name] = r["kernel_ms"] * 1e3
    kb = costmodel.kernel_bytes(cfg, w.batch, w.ctx + warmup + steps // 2)
    out = {}
    for name in ("qkv", "attention", "o_proj", "gate_up", "down"):
        t = us[name] + (us["attn_merge"] if name == "attention" else 0.0)
        gbs = kb[name] / (t / 1e6) / 1e9
        out[name] = {"us": round(t, 2), "bytes": int(kb[name]), "achieved_gbs": round(gbs, 1),
                     "frac": round(gbs / PEAK_HBM_GBS, 4)}
    out["attention"]["score_us"] = round(us["attention"], 2)
    out["attention"]["merge_us"] = round(us["attn_merge"], 2)
    block_us = sum(v["us"] for v in out.values())
    block_bytes = sum(v["bytes"] for v in out.values())
    out["block"] = {"us": round(block_us, 2), "bytes": int(block_bytes),
                    "frac": round(block_bytes / (block_us / 1e6) / 1e9 / PEAK_HBM_GBS, 4)}
    return out


def batched_workload(name, warmup, policy, repeats=1):
    """One batched workload (rerouted every step): its own synthetic model,
    cache and budgets; tokens/s and the step's HBM fraction."""
    import torch
    from paper_2606_09514_amd import lib as blib
    from paper_2606_09514_amd import synth

    w = synth.WORKLOADS[name]
    cfg = synth.model_config(w.shape, w.dtype, w.ctx + warmup + w.steps + 1)
    log(f"generating weights and KV cache for {w.name}")
    W = synth.model_weights(cfg, seed=0, device="cuda", omega=w.omega)
    dk, dv = synth.kv_cache(cfg, w.batch, w.ctx, seed=1, device="cuda")
    x0 = synth.hidden_inputs(w.batch, cfg["d_model"], seed=2, device="cuda")
    model = blib.Model(cfg, W, max_batch=w.batch)
    model.set_launch_policy(policy)
    hip = blib.HipEvents()
    ks = synth.budgets(w, seed=1) if w.mixed else [w.budgets[0]] * w.batch
    r = run_budget(model, cfg, w, dk, dv, x0, ks, w.steps, warmup, hip, 0, repeats=repeats)
    log(f"{w.name}: {r['tokens_per_s']:.1f} tokens/s, {r['ms_per_step']:.3f} ms/step "
        f"(p50 {r['step_ms_p50']:.3f}, p90 {r['step_ms_p90']:.3f}), "
        f"{r['step_hbm_frac'] * 100:.1f}% of HBM roofline; runs "
        + ", ".join(f"{v:.1f}" for v in r["run_tokens_per_s"]) + " tokens/s")
    model.close()
    del model, W, dk, dv, x0
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return {"batch": w.batch, "ctx": w.ctx, "steps": w.steps, "warmup": warmup,
            "k": "mixed " + "/".join(map(str, w.budgets)) if w.mixed else w.budgets[0],
            "mean_k": round(r["mean_k"], 2), "tokens_per_s": round(r["tokens_per_s"], 2),
            "ms_per_step": round(r["ms_per_step"], 4), "step_ms_p50": round(r["step_ms_p50"], 4),
            "step_ms_p90": round(r["step_ms_p90"], 4), "bytes_per_step": int(r["bytes_per_step"]),
            "step_hbm_frac": round(r["step_hbm_frac"], 4), "layers_used": r["layers_used"],
            "distinct_routes": r["distinct_routes"],
            "run_tokens_per_s": [round(v, 2) for v in r["run_tokens_per_s"]],
            "median_tokens_per_s": round(r["median_tokens_per_s"], 2),
            "path_grouping": {"route_groups_per_step": r["route_groups"],
                              "block_runs_per_path_sub_batches": r["per_path_blocks"],
                              "block_runs_per_block_compaction": r["layers_used"]}}


BATCHED = ["llama3_8b_b32_ctx4096_mixed", "qwen2_7b_b64_ctx8192", "mha_13b_b96_ctx2048_mixed"]


def cpu_baseline(cfg, W, dk, dv, x0, k, ctx, budget_s=12.0):
    """The oracle on the host cores: decode steps of sequence 0 of the same
    workload until about budget_s seconds of CPU work (at least one)."""
    import numpy as np
    import torch

    import oracle
    from paper_2606_09514_amd import synth

    log("cpu_baseline: copying weights and sequence 0's cache to the host")
    layers = [{n: synth.storage_numpy(t) for n, t in lw.items()} for lw in W["layers"]]
    dm = {n: (synth.storage_numpy(t) if torch.is_tensor(t) else t) for n, t in W["dm"].items()}
    orc = oracle.Oracle(cfg, layers, dm)
    hk = synth.storage_numpy(dk[:, 0]).copy()
    hv = synth.storage_numpy(dv[:, 0]).copy()
    x = x0[0].cpu().numpy()
    L = cfg["n_layers"]
    n, t0 = 0, time.perf_counter()
    while True:
        h, *_ = orc.decode_seq([hk[l] for l in range(L)], [hv[l] for l in range(L)],
                               ctx + n, k, x)
        x = h.astype(np.float32)
        n += 1
        el = time.perf_counter() - t0
        log(f"cpu_baseline: oracle step {n} done, {el:.1f} s")
        if el >= budget_s or n >= 8:
            break
    return dict(value=n / el, unit="tokens/s", cores=oracle.num_threads(), kind="oracle",
                sample=f"{n} decode step(s) of sequence 0 at k={k}, ctx {ctx}, "
                       f"same weights and cache, oracle in double precision")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--skip-kv", choices=["zero", "mask"], default="zero",
                    help="KV of skipped blocks: zero-filled (the paper's) or masked")
    ap.add_argument("--router-ctx", choices=["kv", "k", "v", "k+v"], default="kv",
                    help="router context features")
    ap.add_argument("--start-layer", type=int, default=1,
                    help="router start layer S: blocks 0..S-1 always run, S..L-2 are routable")
    ap.add_argument("--pool", choices=["scan", "running"], default="scan",
                    help="router pool: sum the first block's rows every step, or keep "
                         "running sums across steps")
    ap.add_argument("--auto-budget", action="store_true",
                    help="budget-free steps: a random-init Budget Predictor picks k")
    ap.add_argument("--prefill", action="store_true",
                    help="time the routed prefill of a prompt of the workload's context length "
                         "at each budget and the dense one, instead of decode steps")
    ap.add_argument("--steps", type=int, default=128)
    ap.add_argument("--repeats", type=int, default=3,
                    help="timed runs per budget: the first gives every figure, all of them the "
                         "median tokens/s (median_tokens_per_s)")
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="llama3_8b_b1_ctx2048")
    ap.add_argument("--budgets", default=None, help="comma list of k (default: the workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--policy", default="auto", choices=["auto", "device", "host"],
                    help="launch policy of the routable blocks")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a 1 GiB device copy first (HBM counter calibration)")
    ap.add_argument("--batched", default="all",
                    help="batched workloads timed after the headline for per_workload: 'all', "
                         "'none' or a comma list of workload names")
    ap.add_argument("--no-per-kernel", action="store_true",
                    help="skip the live per-kernel timing passes of the last block")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the library runs the decode step on one GPU; "
              f"--gpus {args.gpus} is not supported (sharding is design-only)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_09514_amd import lib as blib
    from paper_2606_09514_amd import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    blib.lib()                     # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    w = synth.WORKLOADS[args.workload]
    budgets = [int(b) for b in args.budgets.split(",")] if args.budgets else list(w.budgets)
    cfg = synth.model_config(w.shape, w.dtype, w.ctx + args.warmup + args.steps + 1)
    cfg["router_ctx"] = args.router_ctx
    cfg["start_layer"] = args.start_layer

    if args.copy_calibration:
        a = torch.empty(1 << 28, dtype=torch.float32, device="cuda")   # 1 GiB
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        log("copy calibration: 3 x 1 GiB device copies done")

    log(f"generating weights and KV cache for {w.name}")
    W = synth.model_weights(cfg, seed=0, device="cuda", omega=w.omega)
    dk, dv = synth.kv_cache(cfg, w.batch, w.ctx, seed=1, device="cuda")
    x0 = synth.hidden_inputs(w.batch, cfg["d_model"], seed=2, device="cuda")
    torch.cuda.synchronize()
    model = blib.Model(cfg, W, max_batch=w.batch)
    model.set_launch_policy({"auto": blib.LAUNCH_AUTO, "device": blib.LAUNCH_DEVICE_ROUTED,
                             "host": blib.LAUNCH_HOST_ROUTED}[args.policy])
    hip = blib.HipEvents()
    exec_map = None
    if args.skip_kv == "mask":
        # every cached position ran every block (a dense prefill)
        exec_map = torch.zeros((cfg["n_layers"], w.batch, cfg["max_ctx"]), dtype=torch.uint8,
                               device="cuda")
        exec_map[:, :, :w.ctx] = 1
    if args.auto_budget:
        pw = synth.predictor_weights(cfg, cfg["dm_hidden"], seed=3, device="cuda")
        model.set_budget_predictor(pw)

    if args.prefill:
        Lm = synth.n_mid(cfg)
        ks_list = sorted(set(budgets) | {Lm}) if not w.mixed else [Lm]
        pf = run_prefill(model, cfg, w, dk, dv, ks_list, reps=3, warmup=1)
        dense = pf[str(Lm)]["ms_per_prefill"]
        for r in pf.values():
            r["speedup_vs_dense"] = round(dense / r["ms_per_prefill"], 3)
        head_k = ks_list[0]
        print(json.dumps({
            "metric": "routed prefill tokens/s at budget k (1 GPU)",
            "value": pf[str(head_k)]["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1,
            "higher_is_better": True, "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": w.name, "prompt_tokens": w.ctx, "batch": w.batch, "k": head_k,
                       "router_ctx": args.router_ctx},
            "per_budget": pf}), flush=True)
        model.close()
        return

    runs = {}
    for i, k in enumerate(budgets if not (w.mixed or args.auto_budget) else [None]):
        ks = synth.budgets(w, seed=1) if w.mixed else [k] * w.batch
        if args.auto_budget:
            ks = None
        # the running pool's sums follow the positions forward: one run
        r = run_budget(model, cfg, w, dk, dv, x0, ks, args.steps, args.warmup, hip, 0, exec_map,
                       running_pool=args.pool == "running",
                       repeats=1 if args.pool == "running" else args.repeats)
        name = "auto" if args.auto_budget else "mixed" if w.mixed else str(k)
        runs[name] = r
        log(f"k={name}: {r['tokens_per_s']:.1f} tokens/s, {r['ms_per_step']:.3f} ms/step "
            f"(p50 {r['step_ms_p50']:.3f}, p90 {r['step_ms_p90']:.3f}), "
            f"{r['step_hbm_frac'] * 100:.1f}% of HBM roofline, gate_up {r['kernel_ms'] * 1e3:.1f} us, "
            f"host CPU {r['host_cpu_ms_per_step']:.3f} ms/step; runs "
            + ", ".join(f"{v:.1f}" for v in r["run_tokens_per_s"]) + " tokens/s")

    head = runs[next(iter(runs))]
    head_k = budgets[0] if not (w.mixed or args.auto_budget) else None
    for r in runs.values():
        r.pop("hidden", None)
    d, f = cfg["d_model"], cfg["d_ffn"]
    s = 2 if w.dtype == "bf16" else 4
    # algorithmic bytes of one gate/up launch: weights, input rows, output rows
    gate_up_bytes = 2 * f * d * s + w.batch * d * 4 + w.batch * f * 4
    achieved = gate_up_bytes / (head["kernel_ms"] / 1e3) / 1e9

    kernels = None
    if not args.no_per_kernel and head["ks"] is not None:
        kernels = per_kernel(model, cfg, w, dk, dv, x0, head["ks"], hip)
        log("per-kernel (last block): " + ", ".join(
            f"{n} {v['us']:.1f} us {v['frac'] * 100:.0f}%" for n, v in kernels.items()))

    cpu = None
    if not args.no_cpu_baseline and head["ks"] is not None and args.skip_kv == "zero":
        cpu = cpu_baseline(cfg, W, dk, dv, x0, head["ks"][0], w.ctx)

    policy = {"auto": blib.LAUNCH_AUTO, "device": blib.LAUNCH_DEVICE_ROUTED,
              "host": blib.LAUNCH_HOST_ROUTED}[args.policy]
    batched = []
    if args.batched != "none" and w.name == "llama3_8b_b1_ctx2048" and args.skip_kv == "zero" \
            and not args.auto_budget and args.router_ctx == "kv" and args.start_layer == 1 \
            and args.pool == "scan":
        batched = BATCHED if args.batched == "all" else args.batched.split(",")
    per_workload = {}
    if batched:
        model.close()
        del model, W, dk, dv, x0
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        for name in batched:
            per_workload[name] = batched_workload(name, args.warmup, policy, args.repeats)

    out = {
        "metric": "routed-decode tokens/s at budget k (1 GPU); % of HBM roofline",
        "value": round(head["tokens_per_s"], 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "shape": w.shape, "batch": w.batch, "ctx": w.ctx,
                   "k": head_k if head_k is not None else ("predicted" if args.auto_budget
                                                              else "mixed"),
                   "skip_kv": args.skip_kv, "router_ctx": args.router_ctx, "pool": args.pool,
                   "start_layer": args.start_layer,
                   "weights_kv": w.dtype, "accumulate": "f32", "omega": w.omega,
                   "launch_policy": args.policy,
                   "parallelism": "none (1 GPU)"},
        "per_budget": {n: {"tokens_per_s": round(r["tokens_per_s"], 2),
                           "ms_per_step": round(r["ms_per_step"], 4),
                           "step_ms_p50": round(r["step_ms_p50"], 4),
                           "step_ms_p90": round(r["step_ms_p90"], 4),
                           "bytes_per_step": int(r["bytes_per_step"]),
                           "step_hbm_frac": round(r["step_hbm_frac"], 4),
                           "layers_used": r["layers_used"],
                           "distinct_routes": r["distinct_routes"],
                           "mean_k": round(r["mean_k"], 2),
                           "gate_up_us": round(r["kernel_ms"] * 1e3, 2),
                           "run_tokens_per_s": [round(v, 2) for v in r["run_tokens_per_s"]],
                           "median_tokens_per_s": round(r["median_tokens_per_s"], 2),
                           "host_cpu_ms_per_step": round(r["host_cpu_ms_per_step"], 3)}
                       for n, r in runs.items()},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": measured_traffic() if w.name == "llama3_8b_b1_ctx2048" else None,
                     "kernel": "gemv gate_up+SwiGLU (block 0)",
                     "bytes_per_launch": gate_up_bytes,
                     "launch_us": round(head["kernel_ms"] * 1e3, 2)},
        "per_kernel": kernels,
        "per_workload": per_workload or None,
        "cpu_baseline": cpu,
    }
    if not batched:
        model.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
