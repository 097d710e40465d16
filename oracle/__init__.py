"""TEST INFRASTRUCTURE ONLY: Python access to the CPU reference ("oracle").

The oracle is a plain double-precision C implementation of BUDDY's
budget-routed decode step (arXiv 2606.09514; Sec. 3.1 Eq. 1, Sec. 4.2 Eq. 2,
Sec. 4.3, App. C.1, Sec. 6 limitations).  Only the tests, the smoke check and
the benchmark's CPU-baseline leg may import this package; the product path
never does, and nothing here imports the product package.

Storage arrays are numpy: bf16 as ``np.uint16`` bit patterns, fp32 as
``np.float32``.  A sequence's cache for one layer is ``[n_kv][max_ctx][hd]``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "buddy_oracle.c")

ACTS = {"silu": 0, "gelu": 1}
DTYPES = {"f32": 0, "bf16": 1}
CTXS = {"kv": 0, "k": 1, "v": 2, "k+v": 3}


def build() -> str:
    """Compile the oracle with gcc (no fast-math, no FP contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-ffp-contract=off", "-fopenmp",
           "-fPIC", "-shared", _SRC, "-o", _SO + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_SO + ".tmp", _SO)
    return _SO


class _Config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ffn", C.c_int32),
                ("dm_hidden", C.c_int32), ("dm_act", C.c_int32), ("dtype", C.c_int32),
                ("max_ctx", C.c_int32), ("rms_eps", C.c_double), ("rope_theta", C.c_double),
                ("router_ctx", C.c_int32), ("start_layer", C.c_int32)]


class _Layer(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("attn_norm", "wqkv", "wo", "mlp_norm", "wgate_up", "wdown")]


class _DM(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("b1", C.c_void_p), ("w2", C.c_void_p),
                ("b2", C.c_void_p), ("prior", C.c_void_p), ("omega", C.c_double)]


class _Pred(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("b1", C.c_void_p), ("w2", C.c_void_p),
                ("b2", C.c_void_p), ("hidden", C.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = C.CDLL(_SO)
        vp, i32, dp = C.c_void_p, C.c_int32, C.POINTER(C.c_double)
        L.orc_bf16_from_double.argtypes = [C.c_double]
        L.orc_bf16_from_double.restype = C.c_uint16
        L.orc_rmsnorm.argtypes = [C.POINTER(_Config), vp, vp, vp]
        L.orc_rope.argtypes = [C.POINTER(_Config), vp, i32]
        L.orc_block.argtypes = [C.POINTER(_Config), C.POINTER(_Layer), vp, vp, i32, vp]
        L.orc_pool.argtypes = [C.POINTER(_Config), vp, vp, i32, vp]
        L.orc_dm_scores.argtypes = [C.POINTER(_Config), C.POINTER(_DM), vp, vp]
        L.orc_topk.argtypes = [vp, i32, i32, vp, dp]
        L.orc_topk.restype = C.c_int
        L.orc_decode_seq.argtypes = [C.POINTER(_Config), C.POINTER(_Layer), C.POINTER(_DM),
                                     vp, vp, i32, i32, vp, vp, vp, vp, vp, dp,
                                     C.POINTER(C.c_int32)]
        L.orc_decode_seq.restype = C.c_int
        L.orc_predict_budget.argtypes = [C.POINTER(_Config), C.POINTER(_Pred), vp, vp, dp]
        L.orc_predict_budget.restype = i32
        L.orc_decode_seq_auto.argtypes = [C.POINTER(_Config), C.POINTER(_Layer), C.POINTER(_DM),
                                          C.POINTER(_Pred), vp, vp, vp, i32, vp, vp,
                                          C.POINTER(C.c_int32), vp, dp, vp, vp, dp,
                                          C.POINTER(C.c_int32)]
        L.orc_decode_seq_auto.restype = C.c_int
        L.orc_prefill_seq.argtypes = [C.POINTER(_Config), C.POINTER(_Layer), C.POINTER(_DM),
                                      vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, dp]
        L.orc_prefill_seq.restype = C.c_int
        L.orc_prior_normalize.argtypes = [vp, i32, i32, C.c_double, vp]
        L.orc_group_by_route.argtypes = [vp, i32, i32, vp, vp]
        L.orc_group_by_route.restype = i32
        L.orc_context_dim.argtypes = [C.POINTER(_Config)]
        L.orc_context_dim.restype = C.c_int
        L.orc_router_context.argtypes = [C.POINTER(_Config), vp, vp, i32, vp, vp]
        L.orc_block_ex.argtypes = [C.POINTER(_Config), C.POINTER(_Layer), vp, vp, i32, vp, vp]
        L.orc_decode_seq_ex.argtypes = [C.POINTER(_Config), C.POINTER(_Layer), C.POINTER(_DM),
                                        vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, dp,
                                        C.POINTER(C.c_int32)]
        L.orc_decode_seq_ex.restype = C.c_int
        L.orc_num_threads.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _need(a, dtype, name):
    if not (isinstance(a, np.ndarray) and a.dtype == dtype and a.flags.c_contiguous):
        raise TypeError(f"{name}: expected a C-contiguous {np.dtype(dtype).name} array")
    return a


def bf16_from_double(x: float) -> int:
    return int(lib().orc_bf16_from_double(float(x)))


def prior_normalize(raw, kind: int, winsor: float = 0.0):
    """App. B prior normalisation then Eq. 2 (kind 0 perplexity increase,
    1 Taylor/Fisher, 2 cosine similarity); float64."""
    r = np.ascontiguousarray(raw, dtype=np.float64)
    out = np.empty(r.shape[0], dtype=np.float64)
    lib().orc_prior_normalize(_ptr(r), int(r.shape[0]), int(kind), float(winsor), _ptr(out))
    return out


def group_by_route(mask):
    """Batch-level path grouping of mask [B][n] (nonzero = run): (perm [B],
    starts [n_groups + 1]) as int32 arrays."""
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    B, n = m.shape
    perm = np.zeros(max(B, 1), dtype=np.int32)
    starts = np.zeros(B + 1, dtype=np.int32)
    g = lib().orc_group_by_route(_ptr(m), int(B), int(n), _ptr(perm), _ptr(starts))
    if g < 0:
        raise ValueError("oracle rejected the arguments")
    return perm[:B], starts[:g + 1]


def num_threads() -> int:
    return int(lib().orc_num_threads())


class Oracle:
    """Holds a model (weights as numpy storage arrays) for the C oracle.

    cfg keys: n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn,
    dm_hidden, dm_act ('silu'|'gelu'), dtype ('f32'|'bf16'), max_ctx,
    rms_eps, rope_theta, router_ctx ('kv'|'k'|'v'|'k+v', default 'kv'),
    start_layer (default 1).  layers: list of dicts with attn_norm, wqkv, wo,
    mlp_norm, wgate_up, wdown.  dm: dict with w1, b1, w2, b2, prior (float32
    or None) and omega.
    """

    def __init__(self, cfg: dict, layers: list, dm: dict | None):
        self.cfg = dict(cfg)
        self.sdt = np.uint16 if cfg["dtype"] == "bf16" else np.float32
        self._c = _Config(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                          cfg["head_dim"], cfg["d_ffn"], cfg.get("dm_hidden", 0),
                          ACTS[cfg.get("dm_act", "silu")], DTYPES[cfg["dtype"]],
                          cfg["max_ctx"], float(cfg["rms_eps"]), float(cfg["rope_theta"]),
                          CTXS[cfg.get("router_ctx", "kv")], int(cfg.get("start_layer", 1)))
        self._keep = []
        arr = (_Layer * len(layers))()
        for i, lw in enumerate(layers):
            for n in _Layer._fields_:
                a = _need(lw[n[0]], self.sdt, n[0])
                self._keep.append(a)
                setattr(arr[i], n[0], a.ctypes.data)
        self._layers = arr
        self._dm = None
        if dm is not None:
            d = _DM()
            for n in ("w1", "b1", "w2", "b2"):
                a = _need(dm[n], self.sdt, n)
                self._keep.append(a)
                setattr(d, n, a.ctypes.data)
            pr = dm.get("prior")
            if pr is not None:
                pr = _need(pr, np.float32, "prior")
                self._keep.append(pr)
                d.prior = pr.ctypes.data
            d.omega = float(dm.get("omega", 0.0))
            self._dm = d
        self._pred = None

    def set_predictor(self, pred: dict | None):
        """Budget Predictor weights {w1 [H][din], b1 [H], w2 [L_mid][H], b2
        [L_mid]} as storage arrays, or None."""
        if pred is None:
            self._pred = None
            return
        p = _Pred()
        for n in ("w1", "b1", "w2", "b2"):
            a = _need(pred[n], self.sdt, n)
            self._keep.append(a)
            setattr(p, n, a.ctypes.data)
        p.hidden = int(pred["w1"].shape[0])
        self._pred = p

    def predict_budget(self, z):
        """(k_hat, logits [L_mid] fp32, best - second best logit)."""
        z = np.ascontiguousarray(z, dtype=np.float64)
        lg = np.empty(self.L_mid, dtype=np.float32)
        margin = C.c_double(0.0)
        k = lib().orc_predict_budget(C.byref(self._c), C.byref(self._pred), _ptr(z), _ptr(lg),
                                     C.byref(margin))
        return int(k), lg, margin.value

    def prefill_seq(self, kcs, vcs, x, k: int, route=None, execs=None):
        """Routed prefill of one prompt x [len][d] into rows 0..len-1 of the
        per-layer caches (modified in place).  Returns (h [len][d], mask,
        scores, margin)."""
        L = self.cfg["n_layers"]
        kp = (C.c_void_p * L)(*[_need(a, self.sdt, "kc").ctypes.data for a in kcs])
        vp = (C.c_void_p * L)(*[_need(a, self.sdt, "vc").ctypes.data for a in vcs])
        ep = None
        if execs is not None:
            ep = (C.c_void_p * L)(*[_need(a, np.uint8, "exec").ctypes.data for a in execs])
        x = np.ascontiguousarray(x, dtype=np.float32)
        n = x.shape[0]
        h = np.empty((n, self.cfg["d_model"]), dtype=np.float64)
        mask = np.zeros(self.L_mid, dtype=np.uint8)
        scores = np.zeros(self.L_mid, dtype=np.float32)
        margin = C.c_double(0.0)
        r = None
        if route is not None:
            r = np.ascontiguousarray(route, dtype=np.uint8)
            mask[:] = r
        rc = lib().orc_prefill_seq(C.byref(self._c), self._layers,
                                   C.byref(self._dm) if self._dm is not None else None,
                                   kp, vp, ep, int(n), int(k), _ptr(r), _ptr(x), _ptr(h),
                                   _ptr(mask), _ptr(scores), C.byref(margin))
        if rc != 0:
            raise ValueError("oracle rejected the arguments")
        return h, mask, scores, margin.value

    def decode_seq_auto(self, kcs, vcs, pos: int, x, execs=None):
        """Decode step without a budget (the predictor picks k).  Returns
        (h, k, logits, predictor margin, mask, scores, margin, n_exec)."""
        L = self.cfg["n_layers"]
        kp = (C.c_void_p * L)(*[_need(a, self.sdt, "kc").ctypes.data for a in kcs])
        vp = (C.c_void_p * L)(*[_need(a, self.sdt, "vc").ctypes.data for a in vcs])
        ep = None
        if execs is not None:
            ep = (C.c_void_p * L)(*[_need(a, np.uint8, "exec").ctypes.data for a in execs])
        x = np.ascontiguousarray(x, dtype=np.float32)
        h = np.empty(self.cfg["d_model"], dtype=np.float64)
        k = C.c_int32(0)
        lg = np.zeros(self.L_mid, dtype=np.float32)
        pm = C.c_double(0.0)
        mask = np.zeros(self.L_mid, dtype=np.uint8)
        scores = np.zeros(self.L_mid, dtype=np.float32)
        margin = C.c_double(0.0)
        n_exec = C.c_int32(0)
        rc = lib().orc_decode_seq_auto(C.byref(self._c), self._layers, C.byref(self._dm),
                                       C.byref(self._pred), kp, vp, ep, int(pos), _ptr(x),
                                       _ptr(h), C.byref(k), _ptr(lg), C.byref(pm), _ptr(mask),
                                       _ptr(scores), C.byref(margin), C.byref(n_exec))
        if rc != 0:
            raise ValueError("oracle rejected the arguments")
        return h, k.value, lg, pm.value, mask, scores, margin.value, n_exec.value

    @property
    def start_layer(self) -> int:
        return int(self.cfg.get("start_layer", 1))

    @property
    def L_mid(self) -> int:
        """Routable blocks S..L-2 (S = start_layer)."""
        return self.cfg["n_layers"] - 1 - self.start_layer

    # -- pieces ---------------------------------------------------------
    def rmsnorm(self, h, g):
        h = np.ascontiguousarray(h, dtype=np.float64)
        out = np.empty_like(h)
        lib().orc_rmsnorm(C.byref(self._c), _ptr(h), _ptr(_need(g, self.sdt, "g")), _ptr(out))
        return out

    def rope(self, x, pos: int):
        x = np.array(x, dtype=np.float64, copy=True)
        lib().orc_rope(C.byref(self._c), _ptr(x), int(pos))
        return x

    def block(self, layer: int, kc, vc, pos: int, h, exec=None):
        """exec: optional uint8 execution map [max_ctx] of this layer's cache
        (positions with 0 are left out of the softmax)."""
        h = np.array(h, dtype=np.float64, copy=True)
        ex = None if exec is None else _need(exec, np.uint8, "exec")
        lib().orc_block_ex(C.byref(self._c), C.byref(self._layers[layer]),
                           _ptr(_need(kc, self.sdt, "kc")), _ptr(_need(vc, self.sdt, "vc")),
                           int(pos), _ptr(h), _ptr(ex))
        return h

    def pool(self, kc, vc, pos: int):
        n = self.cfg["n_kv_heads"] * self.cfg["head_dim"]
        z = np.empty(2 * n, dtype=np.float64)
        lib().orc_pool(C.byref(self._c), _ptr(_need(kc, self.sdt, "kc")),
                       _ptr(_need(vc, self.sdt, "vc")), int(pos), _ptr(z))
        return z

    def context(self, kc, vc, pos: int, h):
        """Router context z of one sequence (pooled first-layer features of
        the configured variant, then h)."""
        z = np.empty(int(lib().orc_context_dim(C.byref(self._c))), dtype=np.float64)
        hh = np.ascontiguousarray(h, dtype=np.float64)
        lib().orc_router_context(C.byref(self._c), _ptr(_need(kc, self.sdt, "kc")),
                                 _ptr(_need(vc, self.sdt, "vc")), int(pos), _ptr(hh), _ptr(z))
        return z

    def dm_scores(self, z):
        z = np.ascontiguousarray(z, dtype=np.float64)
        s = np.empty(self.L_mid, dtype=np.float32)
        lib().orc_dm_scores(C.byref(self._c), C.byref(self._dm), _ptr(z), _ptr(s))
        return s

    @staticmethod
    def topk(scores, k: int):
        s = np.ascontiguousarray(scores, dtype=np.float32)
        m = np.zeros(s.shape[0], dtype=np.uint8)
        margin = C.c_double(0.0)
        rc = lib().orc_topk(_ptr(s), s.shape[0], int(k), _ptr(m), C.byref(margin))
        if rc != 0:
            raise ValueError("k out of range")
        return m, margin.value

    # -- the whole step --------------------------------------------------
    def decode_seq(self, kcs, vcs, pos: int, k: int, x, route=None, execs=None):
        """One decode step of one sequence.  kcs/vcs: per-layer cache arrays
        (modified in place); execs: optional per-layer uint8 execution maps
        [max_ctx] for skipped-KV masking (modified in place).  Returns (h,
        mask, scores, margin, n_exec)."""
        L = self.cfg["n_layers"]
        assert len(kcs) == L and len(vcs) == L
        kp = (C.c_void_p * L)(*[_need(a, self.sdt, "kc").ctypes.data for a in kcs])
        vp = (C.c_void_p * L)(*[_need(a, self.sdt, "vc").ctypes.data for a in vcs])
        x = np.ascontiguousarray(x, dtype=np.float32)
        h = np.empty(self.cfg["d_model"], dtype=np.float64)
        mask = np.zeros(self.L_mid, dtype=np.uint8)
        scores = np.zeros(self.L_mid, dtype=np.float32)
        margin = C.c_double(0.0)
        n_exec = C.c_int32(0)
        r = None
        if route is not None:
            r = np.ascontiguousarray(route, dtype=np.uint8)
            mask[:] = r
        ep = None
        if execs is not None:
            assert len(execs) == L
            ep = (C.c_void_p * L)(*[_need(a, np.uint8, "exec").ctypes.data for a in execs])
        rc = lib().orc_decode_seq_ex(C.byref(self._c), self._layers,
                                     C.byref(self._dm) if self._dm is not None else None,
                                     kp, vp, ep, int(pos), int(k), _ptr(r), _ptr(x), _ptr(h),
                                     _ptr(mask), _ptr(scores), C.byref(margin), C.byref(n_exec))
        if rc != 0:
            raise ValueError("oracle rejected the arguments")
        return h, mask, scores, margin.value, n_exec.value
