"""ctypes binding of libbuddy.so, the C ABI declared in include/buddy.h.

Argument marshalling only: torch tensors are passed as device pointers and
torch's current HIP stream as the stream; every step of the decode path runs
in the library's HIP kernels.  Importing this module does not load the
library; the first call does, and fails loudly when it has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

_SO = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbuddy.so")

OK, EINVAL, ESHAPE, ECAPACITY, ENOMEM, EDEVICE, EUNSUPPORTED = range(7)
F32, BF16 = 0, 1
ACT_SILU, ACT_GELU_ERF = 0, 1
SKIP_KV_ZERO, SKIP_KV_MASK = 0, 1
CTX_KV, CTX_K, CTX_V, CTX_K_PLUS_V = 0, 1, 2, 3
PRIOR_DELTA_PPL, PRIOR_TAYLOR, PRIOR_COSINE = 0, 1, 2
CTX_BY_NAME = {"kv": CTX_KV, "k": CTX_K, "v": CTX_V, "k+v": CTX_K_PLUS_V}
LAUNCH_AUTO, LAUNCH_DEVICE_ROUTED, LAUNCH_HOST_ROUTED = 0, 1, 2
GEMM_TILE_AUTO, GEMM_TILE_128, GEMM_TILE_256, GEMM_TILE_256_SPLIT = 0, 1, 2, 3
KERNEL_QKV, KERNEL_ATTENTION, KERNEL_O_PROJ, KERNEL_GATE_UP, KERNEL_DOWN, KERNEL_ATTN_MERGE = range(6)


class Config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ffn", C.c_int32),
                ("dm_hidden", C.c_int32), ("dm_act", C.c_int32), ("dtype", C.c_int32),
                ("max_batch", C.c_int32), ("max_ctx", C.c_int32),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float), ("router_ctx", C.c_int32),
                ("start_layer", C.c_int32)]


class LayerWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("attn_norm", "wqkv", "wo", "mlp_norm", "wgate_up", "wdown")]


class DMWeights(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("b1", C.c_void_p), ("w2", C.c_void_p),
                ("b2", C.c_void_p), ("prior", C.c_void_p), ("omega", C.c_float)]


class PredictorWeights(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("b1", C.c_void_p), ("w2", C.c_void_p),
                ("b2", C.c_void_p), ("hidden", C.c_int32)]


class KV(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("exec", C.c_void_p),
                ("pool_sum", C.c_void_p), ("pool_rows", C.c_void_p)]


class BuddyError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


_lib = None


def lib():
    """The loaded library; raises when the HIP extension is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            raise RuntimeError(f"libbuddy.so is not built ({_SO}); run "
                               "`python -m paper_2606_09514_amd.build` or __graft_entry__.build()")
        L = C.CDLL(_SO)
        vp, i32, P = C.c_void_p, C.c_int32, C.POINTER
        L.buddy_model_create.argtypes = [P(Config), P(LayerWeights), P(DMWeights), P(vp)]
        L.buddy_model_create.restype = C.c_int
        L.buddy_model_destroy.argtypes = [vp]
        L.buddy_model_destroy.restype = None
        L.buddy_pool_route.argtypes = [vp, P(KV), vp, vp, i32, vp, vp]
        L.buddy_pool_route.restype = C.c_int
        L.buddy_pool_route_noalloc.argtypes = [P(Config), P(DMWeights), P(KV), vp, vp, i32, vp,
                                               vp]
        L.buddy_pool_route_noalloc.restype = C.c_int
        L.buddy_select_topk.argtypes = [vp, vp, i32, i32, vp, vp]
        L.buddy_select_topk.restype = C.c_int
        L.buddy_group_by_route.argtypes = [vp, i32, i32, vp, vp, vp, vp]
        L.buddy_group_by_route.restype = C.c_int
        L.buddy_decode_step.argtypes = [vp, P(KV), vp, vp, vp, i32, i32, vp, vp, vp, vp]
        L.buddy_decode_step.restype = C.c_int
        L.buddy_set_launch_policy.argtypes = [vp, i32]
        L.buddy_set_launch_policy.restype = C.c_int
        L.buddy_set_gemm_tile.argtypes = [vp, i32]
        L.buddy_set_gemm_tile.restype = C.c_int
        L.buddy_set_timing_events.argtypes = [vp, i32, i32, vp, vp, i32]
        L.buddy_set_timing_events.restype = C.c_int
        L.buddy_set_budget_predictor.argtypes = [vp, P(PredictorWeights)]
        L.buddy_predict_budget.argtypes = [vp, P(KV), vp, vp, i32, vp, vp, vp]
        L.buddy_decode_step_auto.argtypes = [vp, P(KV), vp, vp, i32, i32, vp, vp, vp, vp]
        L.buddy_prefill.argtypes = [vp, P(KV), vp, i32, vp, vp, i32, i32, vp, vp, vp, vp]
        L.buddy_prior_normalize.argtypes = [vp, i32, i32, C.c_float, vp]
        L.buddy_prior_normalize.restype = C.c_int
        L.buddy_budget_to_k.argtypes = [C.c_float, i32]
        L.buddy_budget_to_k.restype = i32
        L.buddy_status_string.argtypes = [C.c_int]
        L.buddy_status_string.restype = C.c_char_p
        L.buddy_last_error.argtypes = [vp]
        L.buddy_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _dev(t, name, dtype=None):
    if t is None:
        return None
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.is_contiguous()):
        raise TypeError(f"{name}: expected a contiguous device tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    return t.data_ptr()


def _host_i32(values):
    arr = (C.c_int32 * max(len(values), 1))(*[int(v) for v in values])
    return arr


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _raise(rc: int, handle=None):
    if rc != OK:
        L = lib()
        msg = L.buddy_status_string(rc).decode()
        if handle is not None:
            extra = L.buddy_last_error(handle).decode()
            if extra:
                msg += f" ({extra})"
        raise BuddyError(rc, msg)


def budget_to_k(b: float, n_layers: int) -> int:
    return int(lib().buddy_budget_to_k(float(b), int(n_layers)))


def prior_normalize(raw, kind: int, winsor: float = 0.0, check: bool = True):
    """Host wrapper of buddy_prior_normalize: raw indicator values of the
    routable layers -> fp32 prior p~ (numpy)."""
    import numpy as np
    r = np.ascontiguousarray(raw, dtype=np.float32)
    out = np.zeros(r.shape[0], dtype=np.float32)
    rc = lib().buddy_prior_normalize(r.ctypes.data_as(C.c_void_p), int(r.shape[0]), int(kind),
                                     C.c_float(winsor), out.ctypes.data_as(C.c_void_p))
    if check:
        _raise(rc, None)
    return out if rc == OK else rc


def select_topk(scores: torch.Tensor, k, mask_out: torch.Tensor, stream=None,
                check: bool = True) -> int:
    B, n = (scores.shape[0], scores.shape[1]) if scores.dim() == 2 else (0, 0)
    rc = lib().buddy_select_topk(_dev(scores, "scores", torch.float32), _host_i32(k), B, n,
                                 _dev(mask_out, "mask_out", torch.uint8), _stream(stream))
    if check:
        _raise(rc)
    return rc


def _config(cfg: dict, max_batch: int) -> Config:
    return Config(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                  cfg["head_dim"], cfg["d_ffn"], cfg["dm_hidden"],
                  ACT_GELU_ERF if cfg["dm_act"] == "gelu" else ACT_SILU,
                  BF16 if cfg["dtype"] == "bf16" else F32, int(max_batch), cfg["max_ctx"],
                  float(cfg["rms_eps"]), float(cfg["rope_theta"]),
                  CTX_BY_NAME[cfg.get("router_ctx", "kv")], int(cfg.get("start_layer", 1)))


def _dm_weights(dm: dict, dtype) -> DMWeights:
    return DMWeights(_dev(dm["w1"], "w1", dtype), _dev(dm["b1"], "b1", dtype),
                     _dev(dm["w2"], "w2", dtype), _dev(dm["b2"], "b2", dtype),
                     _dev(dm.get("prior"), "prior", torch.float32), float(dm.get("omega", 0.0)))


def pool_route_noalloc(cfg: dict, dm: dict, max_batch: int, k_cache, v_cache, pos, h_new,
                       scores_out, stream=None, check: bool = True, pool=None) -> int:
    """buddy_pool_route_noalloc: planner scores without a model handle or any
    allocation.  cfg as for Model; dm: the Decision Module's device tensors;
    max_batch: batch capacity of the KV cache layout; pool: running-sum pool
    state (sums, row counts) or None."""
    dtype = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    c = _config(cfg, max_batch)
    d = _dm_weights(dm, dtype)
    ps, pr = pool if pool is not None else (None, None)
    kv = KV(_dev(k_cache, "k_cache", dtype), _dev(v_cache, "v_cache", dtype), None,
            _dev(ps, "pool_sum", torch.float32), _dev(pr, "pool_rows", torch.int32))
    rc = lib().buddy_pool_route_noalloc(C.byref(c), C.byref(d), C.byref(kv), _host_i32(pos),
                                        _dev(h_new, "h_new", torch.float32), len(pos),
                                        _dev(scores_out, "scores_out", torch.float32),
                                        _stream(stream))
    if check:
        _raise(rc)
    return rc


def group_by_route(mask: torch.Tensor, perm_out: torch.Tensor, starts_out: torch.Tensor,
                   n_groups_out: torch.Tensor, stream=None, check: bool = True) -> int:
    """buddy_group_by_route: mask uint8 [B][n] -> perm int32 [B], group starts
    int32 [B + 1], group count int32 [1] (device tensors)."""
    B, n = (mask.shape[0], mask.shape[1]) if mask.dim() == 2 else (0, 0)
    rc = lib().buddy_group_by_route(_dev(mask, "mask", torch.uint8), B, n,
                                    _dev(perm_out, "perm_out", torch.int32),
                                    _dev(starts_out, "starts_out", torch.int32),
                                    _dev(n_groups_out, "n_groups_out", torch.int32), _stream(stream))
    if check:
        _raise(rc)
    return rc


class Model:
    """A model handle over caller-owned device weights.

    cfg: dict with the buddy_config fields (dm_act 'silu'|'gelu', dtype
    'f32'|'bf16', router_ctx 'kv'|'k'|'v'|'k+v', default 'kv', start_layer,
    default 1).  weights: {'layers': [dict of tensors], 'dm': {...}} as
    produced by paper_2606_09514_amd.synth.model_weights on the device.
    """

    def __init__(self, cfg: dict, weights: dict, max_batch: int):
        self.cfg = dict(cfg)
        self.dtype = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
        c = _config(cfg, max_batch)
        self._c = c
        self._keep = weights
        L = cfg["n_layers"]
        arr = (LayerWeights * L)()
        for i, lw in enumerate(weights["layers"]):
            for n, _ in LayerWeights._fields_:
                setattr(arr[i], n, _dev(lw[n], n, self.dtype))
        d = _dm_weights(weights["dm"], self.dtype)
        h = C.c_void_p()
        rc = lib().buddy_model_create(C.byref(c), arr, C.byref(d), C.byref(h))
        _raise(rc)
        self._h = h

    @property
    def L_mid(self) -> int:
        """Routable blocks S..L-2 (S = start_layer, default 1)."""
        return self.cfg["n_layers"] - 1 - int(self.cfg.get("start_layer", 1))

    def close(self):
        if getattr(self, "_h", None):
            lib().buddy_model_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def pool_state(self, device="cuda"):
        """Zeroed running-sum pool state (sums fp32 [max_batch][n_kv][2][hd],
        row counts int32 [max_batch][n_kv]) for the `pool` argument."""
        c = self.cfg
        shape = (self._c.max_batch, c["n_kv_heads"])
        return (torch.zeros(shape + (2, c["head_dim"]), dtype=torch.float32, device=device),
                torch.zeros(shape, dtype=torch.int32, device=device))

    def _kv(self, k_cache, v_cache, exec_map=None, pool=None):
        ps, pr = pool if pool is not None else (None, None)
        return KV(_dev(k_cache, "k_cache", self.dtype), _dev(v_cache, "v_cache", self.dtype),
                  _dev(exec_map, "exec_map", torch.uint8), _dev(ps, "pool_sum", torch.float32),
                  _dev(pr, "pool_rows", torch.int32))

    def decode_step(self, k_cache, v_cache, hidden, pos, k, route_override=None,
                    mask_out=None, scores_out=None, skip_kv: int = SKIP_KV_ZERO,
                    stream=None, check: bool = True, exec_map=None, pool=None) -> int:
        """exec_map: device uint8 [L][max_batch][max_ctx] execution map, for
        skip_kv = SKIP_KV_MASK; pool: running-sum pool state (pool_state())
        or None to sum the first block's rows afresh."""
        kv = self._kv(k_cache, v_cache, exec_map, pool)
        B = len(pos)
        rc = lib().buddy_decode_step(
            self._h, C.byref(kv), _dev(hidden, "hidden", torch.float32), _host_i32(pos),
            _host_i32(k) if k is not None else None, B, int(skip_kv),
            _dev(route_override, "route_override", torch.uint8),
            _dev(mask_out, "mask_out", torch.uint8),
            _dev(scores_out, "scores_out", torch.float32), _stream(stream))
        if check:
            _raise(rc, self._h)
        return rc

    def set_budget_predictor(self, weights: dict | None) -> None:
        """Budget Predictor head {w1, b1, w2, b2} (device tensors kept alive
        by the handle), or None to detach."""
        if weights is None:
            _raise(lib().buddy_set_budget_predictor(self._h, None), self._h)
            self._pred = None
            return
        p = PredictorWeights(*[_dev(weights[n], n, self.dtype) for n in ("w1", "b1", "w2", "b2")],
                             int(weights["w1"].shape[0]))
        _raise(lib().buddy_set_budget_predictor(self._h, C.byref(p)), self._h)
        self._pred = weights

    def predict_budget(self, k_cache, v_cache, pos, h_new, k_out, logits_out=None, stream=None,
                       check: bool = True, pool=None) -> int:
        kv = self._kv(k_cache, v_cache, None, pool)
        rc = lib().buddy_predict_budget(self._h, C.byref(kv), _host_i32(pos),
                                        _dev(h_new, "h_new", torch.float32), len(pos),
                                        _dev(k_out, "k_out", torch.int32),
                                        _dev(logits_out, "logits_out", torch.float32),
                                        _stream(stream))
        if check:
            _raise(rc, self._h)
        return rc

    def decode_step_auto(self, k_cache, v_cache, hidden, pos, k_out=None, mask_out=None,
                         scores_out=None, skip_kv: int = SKIP_KV_ZERO, stream=None,
                         check: bool = True, exec_map=None, pool=None) -> int:
        kv = self._kv(k_cache, v_cache, exec_map, pool)
        rc = lib().buddy_decode_step_auto(
            self._h, C.byref(kv), _dev(hidden, "hidden", torch.float32), _host_i32(pos),
            len(pos), int(skip_kv), _dev(k_out, "k_out", torch.int32),
            _dev(mask_out, "mask_out", torch.uint8), _dev(scores_out, "scores_out", torch.float32),
            _stream(stream))
        if check:
            _raise(rc, self._h)
        return rc

    def prefill(self, k_cache, v_cache, hidden, lens, k, route_override=None, mask_out=None,
                scores_out=None, skip_kv: int = SKIP_KV_ZERO, stream=None, check: bool = True,
                exec_map=None, pool=None) -> int:
        """hidden: device [B][t_stride][d] fp32 (in: prompt inputs, out: last
        block outputs); lens: host prompt lengths; k: host budgets or None
        with route_override."""
        kv = self._kv(k_cache, v_cache, exec_map, pool)
        B = len(lens)
        rc = lib().buddy_prefill(
            self._h, C.byref(kv), _dev(hidden, "hidden", torch.float32), int(hidden.shape[1]),
            _host_i32(lens), _host_i32(k) if k is not None else None, B, int(skip_kv),
            _dev(route_override, "route_override", torch.uint8),
            _dev(mask_out, "mask_out", torch.uint8), _dev(scores_out, "scores_out", torch.float32),
            _stream(stream))
        if check:
            _raise(rc, self._h)
        return rc

    def set_launch_policy(self, policy: int) -> None:
        _raise(lib().buddy_set_launch_policy(self._h, int(policy)), self._h)

    def set_gemm_tile(self, tile: int) -> None:
        _raise(lib().buddy_set_gemm_tile(self._h, int(tile)), self._h)

    def set_timing_events(self, kernel: int, layer: int, starts, stops) -> None:
        """starts/stops: sequences of raw hipEvent_t handles (ints)."""
        n = len(starts)
        a = (C.c_void_p * max(n, 1))(*starts)
        b = (C.c_void_p * max(n, 1))(*stops)
        _raise(lib().buddy_set_timing_events(self._h, int(kernel), int(layer),
                                             a if n else None, b if n else None, n), self._h)

    def pool_route(self, k_cache, v_cache, pos, h_new, scores_out, stream=None,
                   check: bool = True, pool=None) -> int:
        kv = self._kv(k_cache, v_cache, None, pool)
        rc = lib().buddy_pool_route(self._h, C.byref(kv), _host_i32(pos),
                                    _dev(h_new, "h_new", torch.float32), len(pos),
                                    _dev(scores_out, "scores_out", torch.float32),
                                    _stream(stream))
        if check:
            _raise(rc, self._h)
        return rc


class HipEvents:
    """Raw hipEvent_t handles for Model.set_timing_events (HIP runtime calls
    through ctypes; the handles are plain ints)."""

    def __init__(self):
        self.h = C.CDLL("libamdhip64.so")
        self.h.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.h.hipEventSynchronize.argtypes = [C.c_void_p]
        self.h.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.h.hipEventDestroy.argtypes = [C.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = C.c_void_p()
            assert self.h.hipEventCreate(C.byref(e)) == 0
            out.append(e.value)
        return out

    def elapsed_ms(self, a, b):
        rc = self.h.hipEventSynchronize(C.c_void_p(b))
        if rc != 0:
            raise RuntimeError(f"hipEventSynchronize: HIP error {rc}")
        ms = C.c_float()
        rc = self.h.hipEventElapsedTime(C.byref(ms), C.c_void_p(a), C.c_void_p(b))
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime: HIP error {rc}")
        return ms.value

    def destroy(self, evs):
        for e in evs:
            self.h.hipEventDestroy(C.c_void_p(e))
