"""ctypes binding of libupr.so (include/upr.h), argument marshalling only.

The functions keep the C names.  Pointers are passed as Python ints (device
pointers from ``tensor.data_ptr()``, host pointers from numpy arrays); the
``*_t`` helpers below accept torch tensors / numpy arrays and check dtypes,
devices and contiguity before calling into the library.  Every compute step
runs in the library's HIP kernels; there is no Python or CPU fallback: if the
shared library is missing, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libupr.so")

UPR_OK, UPR_ERR_NULL, UPR_ERR_CONFIG, UPR_ERR_OFFSETS, UPR_ERR_CAPACITY = 0, 1, 2, 3, 4
UPR_ERR_WORKSPACE, UPR_ERR_DTYPE, UPR_ERR_HIP, UPR_ERR_WEIGHTS, UPR_ERR_LIMIT = 5, 6, 7, 8, 9
UPR_TOPK_MAX_CANDIDATES = 16384
UPR_F32, UPR_BF16, UPR_BF16_MXFP8 = 0, 1, 2
UPR_MX_IN_F32, UPR_MX_IN_F16, UPR_MX_IN_BF16 = 0, 1, 2

# Every symbol include/upr.h declares.
EXPORTS = (
    "upr_weights_count", "upr_model_create", "upr_model_destroy", "upr_kv_cache_bytes",
    "upr_kv_cache_index", "upr_encode_workspace_bytes", "upr_rank_workspace_bytes",
    "upr_encode_user", "upr_rank_candidates", "upr_rank_candidates_noalloc",
    "upr_status_string", "upr_last_error",
    "upr_profile_enable", "upr_profile_read",
    "upr_heads_weights_count", "upr_heads_create", "upr_heads_destroy",
    "upr_rank_actions_workspace_bytes", "upr_rank_actions", "upr_topk_by_utility",
    "upr_mx_quantize_host", "upr_mx_quantize", "upr_mx_linear",
    "upr_kv_pool_create", "upr_kv_pool_export", "upr_kv_pool_export_file", "upr_kv_pool_open",
    "upr_kv_pool_open_file", "upr_kv_pool_slot", "upr_kv_pool_next_slot", "upr_kv_pool_info",
    "upr_kv_pool_destroy",
)


class upr_config(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("d_ff", ctypes.c_int32), ("dtype", ctypes.c_int32), ("ln_eps", ctypes.c_float)]


class upr_segments(ctypes.Structure):
    _fields_ = [("num_users", ctypes.c_int32), ("offsets_host", ctypes.c_void_p),
                ("offsets_dev", ctypes.c_void_p)]


class upr_kv_cache(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("capacity_rows", ctypes.c_int64)]


class upr_heads_config(ctypes.Structure):
    _fields_ = [("n_actions", ctypes.c_int32), ("hidden", ctypes.c_int32)]


UPR_KV_POOL_MAGIC = 0x50525055
UPR_KV_POOL_MAX_BYTES = (2 << 30) - 1


class upr_kv_pool_handle(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_uint32), ("slots", ctypes.c_int32),
                ("capacity_rows", ctypes.c_int64), ("bytes", ctypes.c_uint64),
                ("cfg", upr_config), ("ipc", ctypes.c_uint8 * 64)]


class upr_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double)]


class UprError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"upr status {status}: {message}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH):
    """Load the shared library (once) and declare every signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with paper_2606_00422_amd/build.py "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
    cfgp, segp, cachep = P(upr_config), P(upr_segments), P(upr_kv_cache)
    sig = {
        "upr_weights_count": (I64, [cfgp]),
        "upr_model_create": (I32, [cfgp, VP, I64, P(VP)]),
        "upr_model_destroy": (None, [VP]),
        "upr_kv_cache_bytes": (SZ, [cfgp, I64]),
        "upr_kv_cache_index": (I64, [cfgp, I64, I32, I32, I32, I64, I32]),
        "upr_encode_workspace_bytes": (SZ, [VP, segp]),
        "upr_rank_workspace_bytes": (SZ, [VP, segp, segp]),
        "upr_encode_user": (I32, [VP, VP, segp, cachep, VP, SZ, VP]),
        "upr_rank_candidates": (I32, [VP, cachep, segp, VP, segp, VP, VP, SZ, VP]),
        "upr_rank_candidates_noalloc": (I32, [VP, cachep, segp, VP, segp, VP, VP]),
        "upr_status_string": (ctypes.c_char_p, [I32]),
        "upr_last_error": (ctypes.c_char_p, []),
        "upr_profile_enable": (I32, [I32]),
        "upr_profile_read": (I32, [P(upr_kernel_stat), I32]),
        "upr_heads_weights_count": (I64, [cfgp, P(upr_heads_config)]),
        "upr_heads_create": (I32, [VP, P(upr_heads_config), VP, I64, P(VP)]),
        "upr_heads_destroy": (None, [VP]),
        "upr_rank_actions_workspace_bytes": (SZ, [VP, VP, segp, segp]),
        "upr_rank_actions": (I32, [VP, VP, cachep, segp, VP, segp, VP, VP, VP, VP, SZ, VP]),
        "upr_topk_by_utility": (I32, [VP, segp, I32, VP, VP, VP]),
        "upr_mx_quantize_host": (I32, [VP, I64, I32, VP, VP]),
        "upr_mx_quantize": (I32, [VP, I32, I64, I32, VP, VP, VP]),
        "upr_mx_linear": (I32, [VP, VP, VP, VP, VP, I64, I32, I32, VP, VP]),
        "upr_kv_pool_create": (I32, [cfgp, I32, I64, P(VP)]),
        "upr_kv_pool_export": (I32, [VP, P(upr_kv_pool_handle)]),
        "upr_kv_pool_export_file": (I32, [VP, ctypes.c_char_p]),
        "upr_kv_pool_open": (I32, [P(upr_kv_pool_handle), P(VP)]),
        "upr_kv_pool_open_file": (I32, [ctypes.c_char_p, P(VP)]),
        "upr_kv_pool_slot": (I32, [VP, I32, cachep]),
        "upr_kv_pool_next_slot": (I32, [VP]),
        "upr_kv_pool_info": (I32, [VP, cfgp, P(I32), P(I64)]),
        "upr_kv_pool_destroy": (None, [VP]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != UPR_OK:
        lib = load()
        raise UprError(status, lib.upr_last_error().decode() or
                       lib.upr_status_string(status).decode())


# ---------------------------------------------------------------------------
# The C calls, same names, plain arguments
# ---------------------------------------------------------------------------

DTYPES = {"f32": UPR_F32, "bf16": UPR_BF16, "bf16_mxfp8": UPR_BF16_MXFP8}


def make_config(d_model, n_heads, n_layers, d_ff, dtype, ln_eps=1e-5) -> upr_config:
    """dtype: "f32", "bf16", "bf16_mxfp8" or a upr_dtype value."""
    if d_model % n_heads:
        raise ValueError("d_model must be a multiple of n_heads")
    code = DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
    return upr_config(d_model, n_heads, d_model // n_heads, n_layers, d_ff, code, ln_eps)


def upr_weights_count(cfg: upr_config) -> int:
    return int(load().upr_weights_count(ctypes.byref(cfg)))


def upr_model_create(cfg: upr_config, weights: np.ndarray) -> int:
    w = np.ascontiguousarray(weights, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(load().upr_model_create(ctypes.byref(cfg), w.ctypes.data, w.size, ctypes.byref(out)))
    return int(out.value)


def upr_model_destroy(model: int) -> None:
    load().upr_model_destroy(model)


def upr_kv_cache_bytes(cfg: upr_config, capacity_rows: int) -> int:
    return int(load().upr_kv_cache_bytes(ctypes.byref(cfg), capacity_rows))


def upr_kv_cache_index(cfg, capacity_rows, layer, kv, head, row, e) -> int:
    return int(load().upr_kv_cache_index(ctypes.byref(cfg), capacity_rows, layer, kv, head, row, e))


def upr_encode_workspace_bytes(model: int, hist: upr_segments) -> int:
    return int(load().upr_encode_workspace_bytes(model, ctypes.byref(hist)))


def upr_rank_workspace_bytes(model: int, hist: upr_segments, cand: upr_segments) -> int:
    return int(load().upr_rank_workspace_bytes(model, ctypes.byref(hist), ctypes.byref(cand)))


def upr_encode_user(model, hist_emb_ptr, hist: upr_segments, cache: upr_kv_cache,
                    ws_ptr, ws_bytes, stream) -> None:
    _check(load().upr_encode_user(model, hist_emb_ptr, ctypes.byref(hist), ctypes.byref(cache),
                                  ws_ptr, ws_bytes, stream))


def upr_rank_candidates(model, cache: upr_kv_cache, hist: upr_segments, cand_emb_ptr,
                        cand: upr_segments, scores_ptr, ws_ptr, ws_bytes, stream) -> None:
    _check(load().upr_rank_candidates(model, ctypes.byref(cache), ctypes.byref(hist), cand_emb_ptr,
                                      ctypes.byref(cand), scores_ptr, ws_ptr, ws_bytes, stream))


UPR_NOALLOC_SCRATCH_BYTES = 64 << 20


def upr_rank_candidates_noalloc(model, cache: upr_kv_cache, hist: upr_segments, cand_emb_ptr,
                                cand: upr_segments, scores_ptr, stream) -> None:
    _check(load().upr_rank_candidates_noalloc(model, ctypes.byref(cache), ctypes.byref(hist),
                                              cand_emb_ptr, ctypes.byref(cand), scores_ptr, stream))


def upr_heads_weights_count(cfg: upr_config, hc: upr_heads_config) -> int:
    return int(load().upr_heads_weights_count(ctypes.byref(cfg), ctypes.byref(hc)))


def upr_heads_create(model: int, hc: upr_heads_config, weights: np.ndarray) -> int:
    w = np.ascontiguousarray(weights, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(load().upr_heads_create(model, ctypes.byref(hc), w.ctypes.data, w.size, ctypes.byref(out)))
    return int(out.value)


def upr_heads_destroy(heads: int) -> None:
    load().upr_heads_destroy(heads)


def upr_rank_actions_workspace_bytes(model: int, heads: int, hist: upr_segments,
                                     cand: upr_segments) -> int:
    return int(load().upr_rank_actions_workspace_bytes(model, heads, ctypes.byref(hist),
                                                       ctypes.byref(cand)))


def upr_rank_actions(model, heads, cache: upr_kv_cache, hist: upr_segments, cand_emb_ptr,
                     cand: upr_segments, utility_weights: np.ndarray, probs_ptr, utility_ptr,
                     ws_ptr, ws_bytes, stream) -> None:
    uw = np.ascontiguousarray(utility_weights, dtype=np.float32)
    _check(load().upr_rank_actions(model, heads, ctypes.byref(cache), ctypes.byref(hist),
                                   cand_emb_ptr, ctypes.byref(cand), uw.ctypes.data, probs_ptr,
                                   utility_ptr, ws_ptr, ws_bytes, stream))


def upr_topk_by_utility(utility_ptr, cand: upr_segments, K: int, rows_ptr, values_ptr,
                        stream) -> None:
    _check(load().upr_topk_by_utility(utility_ptr, ctypes.byref(cand), K, rows_ptr, values_ptr,
                                      stream))


def upr_status_string(status: int) -> str:
    return load().upr_status_string(status).decode()


def upr_last_error() -> str:
    return load().upr_last_error().decode()


def upr_profile_enable(enable: bool) -> None:
    _check(load().upr_profile_enable(1 if enable else 0))


def upr_profile_read() -> dict:
    """{kernel name: (launches, total_ms)} recorded since profiling was enabled."""
    lib = load()
    n = lib.upr_profile_read(None, 0)
    arr = (upr_kernel_stat * max(n, 1))()
    n = lib.upr_profile_read(arr, n)
    return {arr[i].name.decode(): (int(arr[i].launches), float(arr[i].total_ms)) for i in range(n)}


# ---------------------------------------------------------------------------
# Marshalling helpers for torch device tensors (torch supplies memory/streams)
# ---------------------------------------------------------------------------

def segments(offsets_host: np.ndarray, offsets_dev=None) -> upr_segments:
    """Descriptor over a host int32 offsets array and its device copy (a torch
    int32 tensor).  The caller keeps both alive for the duration of the call."""
    if offsets_host.dtype != np.int32 or not offsets_host.flags["C_CONTIGUOUS"]:
        raise TypeError("offsets_host must be a contiguous int32 numpy array")
    dev = 0
    if offsets_dev is not None:
        _check_tensor(offsets_dev, "offsets_dev", "int32")
        dev = offsets_dev.data_ptr()
    return upr_segments(int(offsets_host.shape[0] - 1), offsets_host.ctypes.data, dev)


def _check_tensor(t, name, dtype=None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous")
    if dtype is not None and str(t.dtype) != f"torch.{dtype}":
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")


def upr_mx_quantize_host(x: np.ndarray):
    """Host MXFP8 encoding of x [rows, k] (float32): (codes uint8 [rows, k],
    scales uint8 [rows, k / 32])."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    rows, k = x.shape
    codes = np.empty((rows, k), dtype=np.uint8)
    scales = np.empty((rows, max(k // 32, 0)), dtype=np.uint8)
    _check(load().upr_mx_quantize_host(x.ctypes.data, rows, k, codes.ctypes.data, scales.ctypes.data))
    return codes, scales


def upr_mx_quantize(x, codes, scales, stream=None):
    """Device MXFP8 encoding of the 2-D tensor x (float32 / float16 /
    bfloat16) into uint8 tensors codes [rows, k] and scales [rows, k / 32]."""
    import torch
    kinds = {torch.float32: UPR_MX_IN_F32, torch.float16: UPR_MX_IN_F16,
             torch.bfloat16: UPR_MX_IN_BF16}
    for t, name in ((x, "x"), (codes, "codes"), (scales, "scales")):
        if not (t.is_cuda and t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous GPU tensor")
    if x.dtype not in kinds or codes.dtype != torch.uint8 or scales.dtype != torch.uint8:
        raise ValueError("x must be float32/float16/bfloat16, codes and scales uint8")
    rows, k = x.shape
    if tuple(codes.shape) != (rows, k) or tuple(scales.shape) != (rows, k // 32):
        raise ValueError("codes must be [rows, k] and scales [rows, k / 32]")
    _check(load().upr_mx_quantize(x.data_ptr(), kinds[x.dtype], rows, k, codes.data_ptr(),
                                  scales.data_ptr(), current_stream() if stream is None else stream))


def upr_mx_linear(a_codes, a_scales, w_codes, w_scales, bias, out, stream=None):
    """out [M, N] += A W^T + bias with MXFP8 operands (uint8 GPU tensors
    a_codes [M, K], a_scales [M, K/32], w_codes [N, K], w_scales [N, K/32];
    bias [N] and out float32)."""
    import torch
    M, K = a_codes.shape
    N = w_codes.shape[0]
    for t, shape, dt, name in ((a_codes, (M, K), torch.uint8, "a_codes"),
                               (a_scales, (M, K // 32), torch.uint8, "a_scales"),
                               (w_codes, (N, K), torch.uint8, "w_codes"),
                               (w_scales, (N, K // 32), torch.uint8, "w_scales"),
                               (bias, (N,), torch.float32, "bias"), (out, (M, N), torch.float32, "out")):
        if not (t.is_cuda and t.is_contiguous()) or t.dtype != dt or tuple(t.shape) != shape:
            raise ValueError(f"{name} must be a contiguous GPU {dt} tensor of shape {shape}")
    _check(load().upr_mx_linear(a_codes.data_ptr(), a_scales.data_ptr(), w_codes.data_ptr(),
                                w_scales.data_ptr(), bias.data_ptr(), M, N, K, out.data_ptr(),
                                current_stream() if stream is None else stream))


class KvPool:
    """A cross-process KV-cache pool (upr_kv_pool_*): created here (owner) or
    opened from another process's handle file."""

    def __init__(self, handle: int):
        self.handle = handle

    @classmethod
    def create(cls, cfg: upr_config, slots: int, capacity_rows: int) -> "KvPool":
        out = ctypes.c_void_p()
        _check(load().upr_kv_pool_create(ctypes.byref(cfg), slots, capacity_rows, ctypes.byref(out)))
        return cls(int(out.value))

    @classmethod
    def open_file(cls, path: str) -> "KvPool":
        out = ctypes.c_void_p()
        _check(load().upr_kv_pool_open_file(os.fsencode(path), ctypes.byref(out)))
        return cls(int(out.value))

    @classmethod
    def open(cls, h: upr_kv_pool_handle) -> "KvPool":
        out = ctypes.c_void_p()
        _check(load().upr_kv_pool_open(ctypes.byref(h), ctypes.byref(out)))
        return cls(int(out.value))

    def export(self) -> upr_kv_pool_handle:
        h = upr_kv_pool_handle()
        _check(load().upr_kv_pool_export(self.handle, ctypes.byref(h)))
        return h

    def export_file(self, path: str) -> None:
        _check(load().upr_kv_pool_export_file(self.handle, os.fsencode(path)))

    def slot(self, i: int) -> upr_kv_cache:
        c = upr_kv_cache()
        _check(load().upr_kv_pool_slot(self.handle, i, ctypes.byref(c)))
        return c

    def next_slot(self) -> int:
        return int(load().upr_kv_pool_next_slot(self.handle))

    def info(self):
        cfg, slots, rows = upr_config(), ctypes.c_int32(), ctypes.c_int64()
        _check(load().upr_kv_pool_info(self.handle, ctypes.byref(cfg), ctypes.byref(slots),
                                       ctypes.byref(rows)))
        return cfg, int(slots.value), int(rows.value)

    def close(self):
        if self.handle:
            load().upr_kv_pool_destroy(self.handle)
            self.handle = 0


def current_stream() -> int:
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


class Model:
    """A created model plus the tensor-level encode/rank calls."""

    def __init__(self, cfg: upr_config, weights: np.ndarray):
        self.cfg = cfg
        self.handle = upr_model_create(cfg, weights)
        self.torch_dtype = "bfloat16" if cfg.dtype in (UPR_BF16, UPR_BF16_MXFP8) else "float32"

    def close(self):
        if self.handle:
            upr_model_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def new_cache(self, capacity_rows: int):
        import torch
        dt = torch.bfloat16 if self.cfg.dtype in (UPR_BF16, UPR_BF16_MXFP8) else torch.float32
        c = self.cfg
        cache = torch.zeros((c.n_layers, 2, c.n_heads, capacity_rows, c.head_dim), dtype=dt,
                            device="cuda")
        assert cache.numel() * cache.element_size() == upr_kv_cache_bytes(c, capacity_rows)
        return cache

    def workspace(self, nbytes: int):
        import torch
        return torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")

    def encode(self, hist_emb, hist_off_host, hist_off_dev, cache, ws=None, stream=None):
        _check_tensor(hist_emb, "hist_emb", self.torch_dtype)
        _check_tensor(cache, "cache", self.torch_dtype)
        seg = segments(hist_off_host, hist_off_dev)
        need = upr_encode_workspace_bytes(self.handle, seg)
        if ws is None:
            ws = self.workspace(need)
        kv = upr_kv_cache(cache.data_ptr(), cache.shape[3])
        upr_encode_user(self.handle, hist_emb.data_ptr(), seg, kv, ws.data_ptr(), ws.numel(),
                        current_stream() if stream is None else stream)
        return ws

    def rank(self, cache, hist_off_host, hist_off_dev, cand_emb, cand_off_host, cand_off_dev,
             scores, ws=None, stream=None):
        _check_tensor(cand_emb, "cand_emb", self.torch_dtype)
        _check_tensor(cache, "cache", self.torch_dtype)
        _check_tensor(scores, "scores", "float32")
        hs = segments(hist_off_host, hist_off_dev)
        cs = segments(cand_off_host, cand_off_dev)
        need = upr_rank_workspace_bytes(self.handle, hs, cs)
        if ws is None:
            ws = self.workspace(need)
        kv = upr_kv_cache(cache.data_ptr(), cache.shape[3])
        upr_rank_candidates(self.handle, kv, hs, cand_emb.data_ptr(), cs, scores.data_ptr(),
                            ws.data_ptr(), ws.numel(), current_stream() if stream is None else stream)
        return ws

    def rank_actions(self, heads: "Heads", cache, hist_off_host, hist_off_dev, cand_emb,
                     cand_off_host, cand_off_dev, utility_weights, probs=None, utility=None,
                     ws=None, stream=None):
        """upr_rank_actions on tensors: probs [rows, C] and/or utility [rows]
        (float32 GPU tensors indexed like cand_emb rows)."""
        _check_tensor(cand_emb, "cand_emb", self.torch_dtype)
        _check_tensor(cache, "cache", self.torch_dtype)
        if probs is not None:
            _check_tensor(probs, "probs", "float32")
        if utility is not None:
            _check_tensor(utility, "utility", "float32")
        hs = segments(hist_off_host, hist_off_dev)
        cs = segments(cand_off_host, cand_off_dev)
        need = upr_rank_actions_workspace_bytes(self.handle, heads.handle, hs, cs)
        if ws is None:
            ws = self.workspace(need)
        kv = upr_kv_cache(cache.data_ptr(), cache.shape[3])
        upr_rank_actions(self.handle, heads.handle, kv, hs, cand_emb.data_ptr(), cs,
                         np.asarray(utility_weights, dtype=np.float32),
                         0 if probs is None else probs.data_ptr(),
                         0 if utility is None else utility.data_ptr(),
                         ws.data_ptr(), ws.numel(), current_stream() if stream is None else stream)
        return ws


class Heads:
    """Per-action heads created for a model (upr_heads_create)."""

    def __init__(self, model: Model, n_actions: int, hidden: int, weights: np.ndarray):
        self.cfg = upr_heads_config(n_actions, hidden)
        self.handle = upr_heads_create(model.handle, self.cfg, weights)

    def close(self):
        if self.handle:
            upr_heads_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def topk(utility, cand_off_host, cand_off_dev, K, rows, values=None, stream=None):
    """upr_topk_by_utility on tensors: rows int32 [U, K], values float32 [U, K]."""
    _check_tensor(utility, "utility", "float32")
    _check_tensor(rows, "rows", "int32")
    if values is not None:
        _check_tensor(values, "values", "float32")
    cs = segments(cand_off_host, cand_off_dev)
    upr_topk_by_utility(utility.data_ptr(), cs, int(K), rows.data_ptr(),
                        0 if values is None else values.data_ptr(),
                        current_stream() if stream is None else stream)
