"""Helpers shared by the GPU parity tests: one model held twice, as device
tensors for the HIP library and as host storage arrays for the oracle, and a
step comparator implementing the parity rules (exact routes except below a
1e-3 oracle margin, per-row max relative error of the hidden state, new K/V
rows under the same rule, zero-filled rows exactly zero)."""
import numpy as np
import torch

from oracle import Oracle
from paper_2606_09514_amd import lib as blib
from paper_2606_09514_amd import synth

MARGIN = 1e-3
TOL = {"f32": 1e-4, "bf16": 2e-2}


def host_weights(W):
    layers = [{k: synth.storage_numpy(v) for k, v in lw.items()} for lw in W["layers"]]
    dm = {k: (synth.storage_numpy(v) if torch.is_tensor(v) else v) for k, v in W["dm"].items()}
    return layers, dm


def to_device(W):
    layers = [{k: v.cuda() for k, v in lw.items()} for lw in W["layers"]]
    dm = {k: (v.cuda() if torch.is_tensor(v) else v) for k, v in W["dm"].items()}
    return dict(layers=layers, dm=dm)


class Pair:
    """The same model for the GPU library and the oracle."""

    def __init__(self, shape, dtype, max_ctx, batch, seed=0, omega=0.0, device_gen=False,
                 policy=blib.LAUNCH_AUTO):
        self.cfg = synth.model_config(shape, dtype, max_ctx)
        self.batch = batch
        if device_gen:
            self.Wd = synth.model_weights(self.cfg, seed, "cuda", omega=omega)
        else:
            self.Wd = to_device(synth.model_weights(self.cfg, seed, "cpu", omega=omega))
        layers, dm = host_weights(self.Wd)
        self.orc = Oracle(self.cfg, layers, dm)
        self.gpu = blib.Model(self.cfg, self.Wd, max_batch=batch)
        self.gpu.set_launch_policy(policy)
        self.sdt = np.uint16 if dtype == "bf16" else np.float32
        self.tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        L, nkv, hd = self.cfg["n_layers"], self.cfg["n_kv_heads"], self.cfg["head_dim"]
        self.shape5 = (L, batch, nkv, max_ctx, hd)

    @property
    def L_mid(self):
        return self.orc.L_mid

    @property
    def path(self):
        """Projection path the library takes at this batch: the GEMV (fp32
        activations) up to four sequences or in fp32, the MFMA path beyond."""
        return "mfma" if self.cfg["dtype"] == "bf16" and self.batch > 4 else "gemv"

    def empty_host_cache(self):
        return (np.zeros(self.shape5, dtype=self.sdt), np.zeros(self.shape5, dtype=self.sdt))

    def upload(self, host):
        return torch.from_numpy(host.view(np.int16) if self.sdt == np.uint16 else host) \
            .cuda().view(self.tdt)

    def download(self, dev):
        return synth.storage_numpy(dev)


def f32(a, sdt):
    if sdt == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32)
    return a.astype(np.float32)


def relerr(got, ref):
    return float(np.max(np.abs(got - ref)) / max(float(np.max(np.abs(ref))), 1e-30))


# New K/V rows in bf16 storage.  Both sides round their own fp32 / double
# value of the row once to bf16, so where the two unrounded values differ by
# little the stored values are equal or one bf16 ulp apart.  The unrounded
# values differ by the hidden state's error carried into the projection,
# which is a fraction of the row's scale, not of each entry: hence one ulp
# of the entry plus `rel` times the row's largest magnitude, `rel` the
# larger of a floor per path and twice the sequence's measured hidden-state
# error.  The second term matters at small positions: both sides round the
# new V row to bf16, and where the unrounded values straddle a rounding
# boundary the stored values differ by one ulp; at position 0 the attention
# output is that row itself, so the flip passes whole into the O projection
# and the hidden state entering the later blocks (measured: 6.9e-4 at
# position 0 on the MFMA path, whose 16-bit activations flip more entries
# than the GEMV's fp32 ones, 3.8e-5 at position 4, below 1e-5 beyond).
KV_ULP_REL = {"gemv": 1e-4, "mfma": 1e-4}


def bf16_ulp(x):
    """Spacing of bf16 values at |x| (2^(e-7) for |x| in [2^e, 2^(e+1)))."""
    ax = np.maximum(np.abs(x).astype(np.float64), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(ax)) - 7)


def kv_row_err(g, r, rel):
    """Largest violation ratio of |g - r| <= ulp(max(|g|, |r|)) + rel max|r|
    over a row (<= 1 passes)."""
    g = g.astype(np.float64)
    r = r.astype(np.float64)
    bound = bf16_ulp(np.maximum(np.abs(g), np.abs(r))) + rel * max(float(np.max(np.abs(r))), 1e-30)
    return float(np.max(np.abs(g - r) / bound))


def oracle_step(P, hk, hv, b, pos, k, x, route=None, hx=None):
    """One oracle step of sequence b on views of the host caches (modified);
    hx: host execution maps [L][B][T] for skipped-KV masking (modified)."""
    L = P.cfg["n_layers"]
    kcs = [hk[l, b] for l in range(L)]
    vcs = [hv[l, b] for l in range(L)]
    execs = None if hx is None else [hx[l, b] for l in range(L)]
    return P.orc.decode_seq(kcs, vcs, pos, k, x, route=route, execs=execs)


def gpu_step(P, dk, dv, x, pos, ks, route=None, dx=None, pool=None):
    """One GPU step; dx: device execution map (skipped-KV masking) or None;
    pool: running-sum pool state or None."""
    B = len(pos)
    hidden = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    mask = torch.zeros((B, P.L_mid), dtype=torch.uint8, device="cuda")
    scores = torch.zeros((B, P.L_mid), dtype=torch.float32, device="cuda")
    ro = None if route is None else torch.from_numpy(np.asarray(route, np.uint8)).cuda()
    P.gpu.decode_step(dk, dv, hidden, pos, ks, route_override=ro, mask_out=mask,
                      scores_out=scores, exec_map=dx, pool=pool,
                      skip_kv=blib.SKIP_KV_ZERO if dx is None else blib.SKIP_KV_MASK)
    torch.cuda.synchronize()
    return hidden.cpu().numpy(), mask.cpu().numpy(), scores.cpu().numpy()


def compare_step(P, hk, hv, dk, dv, x, pos, ks, report, hx=None, dx=None, pool=None):
    """Teacher-forced step: the GPU caches (and execution maps hx/dx, with
    masking) hold the oracle's state on entry.  Runs both sides, applies the
    parity rules, and leaves the oracle's post-step state in hk/hv/hx (re-run
    with the GPU's route where the routes legitimately differ).  Returns the
    oracle outputs [B][d]."""
    B = len(pos)
    tol = TOL[P.cfg["dtype"]]
    hg, mg, sg = gpu_step(P, dk, dv, x, pos, ks, dx=dx, pool=pool)
    gk, gv = P.download(dk), P.download(dv)
    gx = None if dx is None else dx.cpu().numpy()
    out = np.zeros((B, P.cfg["d_model"]))
    for b in range(B):
        pre_k = [hk[l, b].copy() for l in range(P.cfg["n_layers"])]
        pre_v = [hv[l, b].copy() for l in range(P.cfg["n_layers"])]
        pre_x = None if hx is None else [hx[l, b].copy() for l in range(P.cfg["n_layers"])]
        h, m, s, margin, n_exec = oracle_step(P, hk, hv, b, pos[b], ks[b], x[b], hx=hx)
        assert n_exec == ks[b] + P.orc.start_layer + 1 and int(m.sum()) == ks[b]
        if not np.array_equal(m, mg[b]):
            assert margin < MARGIN, f"route mismatch at margin {margin} (seq {b})"
            report["margin_mismatches"] += 1
            for l in range(P.cfg["n_layers"]):
                hk[l, b] = pre_k[l]
                hv[l, b] = pre_v[l]
                if hx is not None:
                    hx[l, b] = pre_x[l]
            h, *_ = oracle_step(P, hk, hv, b, pos[b], ks[b], x[b], route=mg[b], hx=hx)
        if hx is not None:   # the execution map is integer data: exact
            assert np.array_equal(gx[:, b], hx[:, b]), f"execution map differs (seq {b})"
        assert int(mg[b].sum()) == ks[b]
        err = relerr(hg[b], h)
        report["max_hidden_err"] = max(report["max_hidden_err"], err)
        assert err < tol, f"hidden rel err {err} (seq {b}, pos {pos[b]})"
        # new K/V rows of every block, same rule; skipped blocks exactly zero
        run = np.concatenate([[1] * P.orc.start_layer, mg[b], [1]])
        for l in range(P.cfg["n_layers"]):
            for ref, got in ((hk, gk), (hv, gv)):
                r = f32(ref[l, b, :, pos[b]], P.sdt)
                g = f32(got[l, b, :, pos[b]], P.sdt)
                if run[l]:
                    e = relerr(g, r)
                    report["max_kv_err"] = max(report["max_kv_err"], e)
                    assert e < tol, f"new KV row err {e} (layer {l}, seq {b})"
                    if P.sdt == np.uint16:
                        v = kv_row_err(g, r, max(KV_ULP_REL[P.path], 2 * err))
                        report["max_kv_ulp_ratio"] = max(report.get("max_kv_ulp_ratio", 0.0), v)
                        assert v <= 1.0, f"new KV row beyond one bf16 ulp: {v} (layer {l}, seq {b})"
                else:
                    assert np.all(g == 0) and np.all(r == 0)
        out[b] = h
    return out, mg
