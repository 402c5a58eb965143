"""ctypes binding of libmoe (include/moe.h): argument marshalling only.

Every function takes torch tensors that live on the GPU, checks dtype, shape
and contiguity, allocates missing outputs with torch (device memory only) and
calls the C entry point of the same name on torch's current stream. There is
no CPU path: if libmoe.so is missing or a tensor is not on the GPU, the call
raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoe.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP = range(5)
MOE_F32, MOE_BF16 = 0, 1
MAX_EXPERTS, MAX_TOPK = 256, 16

EXPORTED = ("moe_status_string", "moe_abi_version", "moe_gate_topk", "moe_expert_histogram_scan",
            "moe_permute", "moe_grouped_swiglu_ffn", "moe_unpermute_combine", "moe_load_sweep",
            "moe_fit_latency_model", "moe_place_greedy", "moe_place_incremental", "moe_placement_cost",
            "moe_window_push", "moe_drift_distance", "moe_mx_quantize", "moe_grouped_swiglu_mx",
            "moe_grouped_gemm_mx", "moe_grouped_swiglu_ffn_mx", "moe_load_sweep_mx",
            "moe_grouped_swiglu_ffn_gather", "moe_grouped_swiglu_ffn_noalloc", "moe_ffn_scratch_bytes")


class MoeError(RuntimeError):
    def __init__(self, fn, status, text):
        super().__init__(f"{fn} failed: status {status} ({text})")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t
_PSZ = ctypes.POINTER(ctypes.c_size_t)


def load_library(path: str = LIB_PATH):
    """Load libmoe.so (built in-tree by ``paper_2606_00735_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -m paper_2606_00735_amd.build`")
    L = ctypes.CDLL(path)
    L.moe_status_string.restype = ctypes.c_char_p
    L.moe_status_string.argtypes = [_I]
    L.moe_abi_version.restype = _I
    L.moe_abi_version.argtypes = []
    L.moe_gate_topk.restype = _I
    L.moe_gate_topk.argtypes = [_P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _PSZ, _P]
    L.moe_expert_histogram_scan.restype = _I
    L.moe_expert_histogram_scan.argtypes = [_P, _I, _I, _I, _P, _I, _P, _P, _P, _PSZ, _P]
    L.moe_permute.restype = _I
    L.moe_permute.argtypes = [_P, _P, _P, _P, _SZ, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P]
    L.moe_grouped_swiglu_ffn.restype = _I
    L.moe_grouped_swiglu_ffn.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P, _P, _PSZ, _P]
    L.moe_grouped_swiglu_ffn_gather.restype = _I
    L.moe_grouped_swiglu_ffn_gather.argtypes = [_P, _P, _I, _I, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P, _P,
                                                _PSZ, _P]
    L.moe_unpermute_combine.restype = _I
    L.moe_unpermute_combine.argtypes = [_P, _P, _P, _I, _I, _I, _I, _I, _P, _P]
    L.moe_load_sweep.restype = _I
    L.moe_load_sweep.argtypes = [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P, _PSZ, _P, _P, _P]
    _D = ctypes.c_double
    L.moe_fit_latency_model.restype = _I
    L.moe_fit_latency_model.argtypes = [_P, _P, _I, _P, _P]
    L.moe_place_greedy.restype = _I
    L.moe_place_greedy.argtypes = [_P, _I, _I, _P, _P, _I, _I, _I, _P, _P, _P, _P]
    L.moe_place_incremental.restype = _I
    L.moe_place_incremental.argtypes = [_P, _I, _I, _P, _P, _I, _I, _D, _I, _P, _P, _P]
    L.moe_placement_cost.restype = _I
    L.moe_placement_cost.argtypes = [_P, _P, _I, _I, _P, _P, _I, _I, _P, _P, _P, _P]
    L.moe_window_push.restype = _I
    L.moe_window_push.argtypes = [_P, _P, _P, _I, _I, _I, _I, _P]
    L.moe_drift_distance.restype = _I
    L.moe_drift_distance.argtypes = [_P, _P, _I, _I, _D, _P, _P, _P]
    L.moe_mx_quantize.restype = _I
    L.moe_mx_quantize.argtypes = [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P]
    L.moe_grouped_swiglu_mx.restype = _I
    L.moe_grouped_swiglu_mx.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P]
    L.moe_grouped_gemm_mx.restype = _I
    L.moe_grouped_gemm_mx.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P]
    L.moe_load_sweep_mx.restype = _I
    L.moe_load_sweep_mx.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P, _PSZ,
                                    _P, _P, _P]
    L.moe_grouped_swiglu_ffn_mx.restype = _I
    L.moe_grouped_swiglu_ffn_mx.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _PSZ,
                                            _P]
    L.moe_grouped_swiglu_ffn_noalloc.restype = _I
    L.moe_grouped_swiglu_ffn_noalloc.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P, _P]
    L.moe_ffn_scratch_bytes.restype = _SZ
    L.moe_ffn_scratch_bytes.argtypes = []
    if L.moe_abi_version() != 3:
        raise RuntimeError("libmoe ABI version mismatch")
    _lib = L
    return L


def _check(fn, status):
    if status != MOE_OK:
        text = load_library().moe_status_string(status).decode()
        raise MoeError(fn, status, text)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, name, dtype=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU (libmoe has no CPU path)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _wrows(t, name, dtype):
    """A batch of weight matrices [B, R, K] whose rows may be padded: a view
    with unit element stride, row stride ld >= K and matrix stride R * ld (as
    the columns [:, :, :K] of a [B, R, ld] tensor). Returns (pointer, ld)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU (libmoe has no CPU path)")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    B, R, K = t.shape
    if t.numel() == 0:  # no experts (or empty matrices): nothing is read
        return ctypes.c_void_p(t.data_ptr()), K
    ld = t.stride(1) if R > 1 else K
    if t.stride(2) != 1 or ld < K or (B > 1 and t.stride(0) != R * ld):
        raise ValueError(f"{name} must be [B, R, K] with unit element stride and rows {ld} apart")
    return ctypes.c_void_p(t.data_ptr()), ld


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise ValueError(f"unsupported dtype {t.dtype}: bf16 or fp32")


def _host_map(expert_map):
    a = np.ascontiguousarray(np.asarray(expert_map, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _ptr_or_null(t, name, dtype=None):
    return ctypes.c_void_p(None) if t is None else _dev(t, name, dtype)


# ---------------------------------------------------------------------------
# The six entry points
# ---------------------------------------------------------------------------
def gate_ws_bytes(T, H, E, dtype):
    """Bytes of the router's optional workspace (0 where it is not used)."""
    L = load_library()
    n = ctypes.c_size_t(0)
    dt = MOE_BF16 if dtype == torch.bfloat16 else MOE_F32
    st = L.moe_gate_topk(None, None, None, T, H, E, 1, dt, None, None, None, None, ctypes.byref(n), None)
    _check("moe_gate_topk", st)
    return n.value


def moe_gate_topk(x, w_router, bias, k, logits=False, ids=None, weights=None, ws=None, use_ws=True):
    """Top-k gating. Returns (ids [T,k] int32, weights [T,k] fp32, logits [T,E] or None).
    ws: the router's workspace (allocated here when needed and not given);
    use_ws=False runs the router without one."""
    L = load_library()
    T, H = x.shape
    E = w_router.shape[0]
    dt = _dtype_code(x)
    if w_router.dtype != x.dtype or tuple(w_router.shape) != (E, H):
        raise ValueError("w_router must be [E, H] with the dtype of x")
    dev = x.device
    ids = torch.empty((T, k), dtype=torch.int32, device=dev) if ids is None else ids
    weights = torch.empty((T, k), dtype=torch.float32, device=dev) if weights is None else weights
    lg = torch.empty((T, E), dtype=torch.float32, device=dev) if logits is True else (
        logits if isinstance(logits, torch.Tensor) else None)
    pws, n = ctypes.c_void_p(None), None
    if use_ws:
        need = gate_ws_bytes(T, H, E, x.dtype)
        if need > 0:
            if ws is None or ws.numel() * ws.element_size() < need:
                ws = torch.empty(need, dtype=torch.uint8, device=dev)
            pws, n = _dev(ws, "ws"), ctypes.c_size_t(ws.numel() * ws.element_size())
    st = L.moe_gate_topk(_dev(x, "x"), _dev(w_router, "w_router"), _ptr_or_null(bias, "bias", torch.float32),
                         T, H, E, k, dt, _ptr_or_null(lg, "logits", torch.float32),
                         _dev(ids, "ids", torch.int32), _dev(weights, "weights", torch.float32), pws,
                         ctypes.byref(n) if n is not None else None, _stream())
    _check("moe_gate_topk", st)
    return ids, weights, lg


def hist_ws_bytes(T, k, E, expert_map_len_local):
    L = load_library()
    n = ctypes.c_size_t(0)
    st = L.moe_expert_histogram_scan(None, T, k, E, None, expert_map_len_local, None, None, None,
                                     ctypes.byref(n), None)
    _check("moe_expert_histogram_scan", st)
    return n.value


def moe_expert_histogram_scan(ids, E, expert_map, ws=None, counts=None, offsets=None):
    """Activation profile. Returns (counts [E], offsets [E_local+1], ws)."""
    L = load_library()
    T, k = ids.shape
    emap, emap_p = _host_map(expert_map)
    if emap.shape != (E,):
        raise ValueError("expert_map must have E entries")
    E_local = int((emap >= 0).sum())
    need = hist_ws_bytes(T, k, E, E_local)
    dev = ids.device
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
    counts = torch.empty(E, dtype=torch.int32, device=dev) if counts is None else counts
    offsets = torch.empty(E_local + 1, dtype=torch.int32, device=dev) if offsets is None else offsets
    n = ctypes.c_size_t(ws.numel() * ws.element_size())
    st = L.moe_expert_histogram_scan(_dev(ids, "ids", torch.int32), T, k, E, emap_p, E_local,
                                     _dev(counts, "counts", torch.int32), _dev(offsets, "offsets", torch.int32),
                                     _dev(ws, "ws"), ctypes.byref(n), _stream())
    _check("moe_expert_histogram_scan", st)
    return counts, offsets, ws


def moe_permute(x, ids, expert_map, ws, M_cap=None, x_perm=None, perm_src=None, dest=None, gather=True):
    """Dispatch. Returns (x_perm [M_cap,H], perm_src [M_cap], dest [T*k]); with
    gather=False only the positions (x_perm is None), for
    moe_grouped_swiglu_ffn_gather."""
    L = load_library()
    T, H = x.shape
    k = ids.shape[1]
    emap, emap_p = _host_map(expert_map)
    E = emap.shape[0]
    E_local = int((emap >= 0).sum())
    M_cap = T * k if M_cap is None else M_cap
    dev = x.device
    if not gather:
        x_perm = None
    elif x_perm is None:
        x_perm = torch.empty((M_cap, H), dtype=x.dtype, device=dev)
    perm_src = torch.empty(M_cap, dtype=torch.int32, device=dev) if perm_src is None else perm_src
    dest = torch.empty(T * k, dtype=torch.int32, device=dev) if dest is None else dest
    st = L.moe_permute(_dev(x, "x"), _dev(ids, "ids", torch.int32), emap_p, _dev(ws, "ws"),
                       ws.numel() * ws.element_size(), T, H, k, E, E_local, M_cap, _dtype_code(x),
                       _ptr_or_null(x_perm, "x_perm", x.dtype), _dev(perm_src, "perm_src", torch.int32),
                       _dev(dest, "dest", torch.int32), _stream())
    _check("moe_permute", st)
    return x_perm, perm_src, dest


def ffn_ws_bytes(E_local, H, I, M_cap, dtype):
    L = load_library()
    n = ctypes.c_size_t(0)
    dt = MOE_BF16 if dtype == torch.bfloat16 else MOE_F32
    st = L.moe_grouped_swiglu_ffn(None, None, None, None, None, E_local, H, I, 0, 0, M_cap, dt, None, None,
                                  ctypes.byref(n), None)
    _check("moe_grouped_swiglu_ffn", st)
    return n.value


def weight_row_stride(K, elem_bytes=2):
    """Row stride (elements) for expert weight rows of K elements of
    `elem_bytes` bytes: rows whose byte length is a multiple of 4 KiB put the
    rows of a weight tile on few HBM channels, so they get 128 bytes of
    padding (whole cache lines); other rows stay dense. Measured for bf16
    weights (H = 4096 or 2048: the decode FFN 6-10 % faster); MXFP8 code
    rows of 4 KiB streamed no faster padded."""
    return K + 128 // elem_bytes if (K * elem_bytes) % 4096 == 0 else K


def pad_weight_rows(w, ld=None):
    """Copy of weights [B, R, K] whose rows are ``ld`` elements apart
    (default ``weight_row_stride``), returned as the view [:, :, :K] of a
    [B, R, ld] tensor; the FFN entry points take such views as they are.
    The padding is zero-filled and never read."""
    B, R, K = w.shape
    ld = weight_row_stride(K, w.element_size()) if ld is None else ld
    if ld == K:
        return w.contiguous()
    buf = torch.zeros((B, R, ld), dtype=w.dtype, device=w.device)
    buf[:, :, :K] = w
    return buf[:, :, :K]


def _ffn_weights(w_gate, w_up, w_down, dtype):
    """Pointers and row strides of the expert weights (w_gate and w_up must
    share their row stride)."""
    pg, ld_gu = _wrows(w_gate, "w_gate", dtype)
    pu, ld_u = _wrows(w_up, "w_up", dtype)
    pd, ld_dn = _wrows(w_down, "w_down", dtype)
    if ld_u != ld_gu:
        raise ValueError("w_gate and w_up must have the same row stride")
    return pg, pu, pd, ld_gu, ld_dn


def moe_grouped_swiglu_ffn(x_perm, w_gate, w_up, w_down, offsets, ws=None, y_perm=None):
    """Grouped SwiGLU FFN over local experts. Returns (y_perm [M_cap,H], ws)."""
    L = load_library()
    M_cap, H = x_perm.shape
    E_local, I, H2 = w_gate.shape
    if H2 != H or tuple(w_up.shape) != (E_local, I, H) or tuple(w_down.shape) != (E_local, H, I):
        raise ValueError("expert weights must be w_gate/w_up [E_local, I, H] and w_down [E_local, H, I]")
    if offsets.numel() != E_local + 1:
        raise ValueError("offsets must have E_local + 1 entries")
    dt = _dtype_code(x_perm)
    need = ffn_ws_bytes(E_local, H, I, M_cap, x_perm.dtype)
    if ws is None:
        ws = torch.zeros(need, dtype=torch.uint8, device=x_perm.device)  # counters start at zero
    y_perm = torch.empty((M_cap, H), dtype=x_perm.dtype, device=x_perm.device) if y_perm is None else y_perm
    n = ctypes.c_size_t(ws.numel() * ws.element_size())
    pg, pu, pd, ld_gu, ld_dn = _ffn_weights(w_gate, w_up, w_down, x_perm.dtype)
    st = L.moe_grouped_swiglu_ffn(_dev(x_perm, "x_perm"), pg, pu, pd,
                                  _dev(offsets, "offsets", torch.int32), E_local, H, I, ld_gu, ld_dn, M_cap, dt,
                                  _dev(y_perm, "y_perm", x_perm.dtype), _dev(ws, "ws"), ctypes.byref(n),
                                  _stream())
    _check("moe_grouped_swiglu_ffn", st)
    return y_perm, ws


def moe_grouped_swiglu_ffn_noalloc(x_perm, w_gate, w_up, w_down, offsets, y_perm):
    """moe_grouped_swiglu_ffn on the library's per-GPU scratch: allocates
    nothing (y_perm [M_cap, H] must be given). Returns y_perm."""
    L = load_library()
    M_cap, H = x_perm.shape
    E_local, I, H2 = w_gate.shape
    if H2 != H or tuple(w_up.shape) != (E_local, I, H) or tuple(w_down.shape) != (E_local, H, I):
        raise ValueError("expert weights must be w_gate/w_up [E_local, I, H] and w_down [E_local, H, I]")
    if offsets.numel() != E_local + 1:
        raise ValueError("offsets must have E_local + 1 entries")
    if tuple(y_perm.shape) != (M_cap, H):
        raise ValueError("y_perm must be [M_cap, H]")
    pg, pu, pd, ld_gu, ld_dn = _ffn_weights(w_gate, w_up, w_down, x_perm.dtype)
    st = L.moe_grouped_swiglu_ffn_noalloc(_dev(x_perm, "x_perm"), pg, pu, pd,
                                          _dev(offsets, "offsets", torch.int32), E_local, H, I, ld_gu, ld_dn, M_cap,
                                          _dtype_code(x_perm), _dev(y_perm, "y_perm", x_perm.dtype), _stream())
    _check("moe_grouped_swiglu_ffn_noalloc", st)
    return y_perm


def moe_grouped_swiglu_ffn_gather(x, perm_src, k, w_gate, w_up, w_down, offsets, ws=None, y_perm=None):
    """The grouped SwiGLU FFN reading row r of its input as x[perm_src[r] // k]
    (bf16). Same results as moe_permute + moe_grouped_swiglu_ffn. Returns
    (y_perm [M_cap,H], ws)."""
    L = load_library()
    T, H = x.shape
    M_cap = perm_src.numel()
    E_local, I, H2 = w_gate.shape
    if H2 != H or tuple(w_up.shape) != (E_local, I, H) or tuple(w_down.shape) != (E_local, H, I):
        raise ValueError("expert weights must be w_gate/w_up [E_local, I, H] and w_down [E_local, H, I]")
    if offsets.numel() != E_local + 1:
        raise ValueError("offsets must have E_local + 1 entries")
    dt = _dtype_code(x)
    need = ffn_ws_bytes(E_local, H, I, M_cap, x.dtype)
    if ws is None:
        ws = torch.zeros(need, dtype=torch.uint8, device=x.device)  # counters start at zero
    y_perm = torch.empty((M_cap, H), dtype=x.dtype, device=x.device) if y_perm is None else y_perm
    n = ctypes.c_size_t(ws.numel() * ws.element_size())
    pg, pu, pd, ld_gu, ld_dn = _ffn_weights(w_gate, w_up, w_down, x.dtype)
    st = L.moe_grouped_swiglu_ffn_gather(_dev(x, "x"), _dev(perm_src, "perm_src", torch.int32), T, k,
                                         pg, pu, pd, _dev(offsets, "offsets", torch.int32),
                                         E_local, H, I, ld_gu, ld_dn, M_cap, dt, _dev(y_perm, "y_perm", x.dtype),
                                         _dev(ws, "ws"), ctypes.byref(n), _stream())
    _check("moe_grouped_swiglu_ffn_gather", st)
    return y_perm, ws


def moe_unpermute_combine(y_perm, weights, dest, T, out=None):
    """Weighted combine back to token order. Returns out [T,H]."""
    L = load_library()
    M_cap, H = y_perm.shape
    k = weights.shape[1]
    out = torch.empty((T, H), dtype=y_perm.dtype, device=y_perm.device) if out is None else out
    st = L.moe_unpermute_combine(_dev(y_perm, "y_perm"), _dev(weights, "weights", torch.float32),
                                 _dev(dest, "dest", torch.int32), T, k, H, M_cap, _dtype_code(y_perm),
                                 _dev(out, "out", y_perm.dtype), _stream())
    _check("moe_unpermute_combine", st)
    return out


def moe_load_sweep(x, w_gate, w_up, w_down, Ms, warmup=3, iters=10, y_scratch=None, ws=None,
                   keep_all=False):
    """Per-expert latency vs token load. Returns (median_us [nM], all_us [nM,iters] or None)."""
    L = load_library()
    n_rot, I, H = w_gate.shape
    Ms = np.ascontiguousarray(np.asarray(Ms, dtype=np.int32))
    nM = len(Ms)
    max_m = int(Ms.max())
    if x.shape[0] < max_m or x.shape[1] != H:
        raise ValueError("x must be [max(Ms), H]")
    dt = _dtype_code(x)
    n = ctypes.c_size_t(0)
    st = L.moe_load_sweep(None, None, None, None, n_rot, H, I, 0, 0, dt, Ms.ctypes.data_as(ctypes.c_void_p), nM,
                          warmup, iters, None, None, ctypes.byref(n), None, None, None)
    _check("moe_load_sweep", st)
    if ws is None:
        ws = torch.zeros(n.value, dtype=torch.uint8, device=x.device)  # counters start at zero
    if y_scratch is None:
        y_scratch = torch.empty((max_m, H), dtype=x.dtype, device=x.device)
    us = np.zeros(nM, np.float32)
    us_all = np.zeros((nM, iters), np.float32) if keep_all else None
    n = ctypes.c_size_t(ws.numel())
    pg, pu, pd, ld_gu, ld_dn = _ffn_weights(w_gate, w_up, w_down, x.dtype)
    st = L.moe_load_sweep(_dev(x, "x"), pg, pu, pd, n_rot, H, I, ld_gu, ld_dn, dt,
                          Ms.ctypes.data_as(ctypes.c_void_p), nM, warmup, iters, _dev(y_scratch, "y_scratch", x.dtype), _dev(ws, "ws"),
                          ctypes.byref(n), us.ctypes.data_as(ctypes.c_void_p),
                          us_all.ctypes.data_as(ctypes.c_void_p) if keep_all else None, _stream())
    _check("moe_load_sweep", st)
    return us, us_all


# ---------------------------------------------------------------------------
# Whole layer: the five stream-ordered calls, no host synchronisation.
# ---------------------------------------------------------------------------
def moe_layer(x, w_router, bias, k, expert_map, w_gate, w_up, w_down, logits=False, bufs=None,
              fuse_gather=False):
    """One GPU's share of the MoE layer; returns a dict of every output.

    ``bufs`` (optional dict) supplies preallocated outputs and workspaces so
    that repeated calls allocate nothing. ``fuse_gather`` (bf16): the FFN
    reads the routed rows of x itself (moe_grouped_swiglu_ffn_gather) and
    x_perm is not built (None in the result); every other output is the same.
    """
    b = {} if bufs is None else bufs
    T = x.shape[0]
    E = w_router.shape[0]
    gws = b.get("gate_ws")
    if gws is None:
        need = gate_ws_bytes(T, x.shape[1], E, x.dtype)
        gws = torch.empty(need, dtype=torch.uint8, device=x.device) if need > 0 else None
    ids, wts, lg = moe_gate_topk(x, w_router, bias, k, logits=logits, ids=b.get("ids"),
                                 weights=b.get("weights"), ws=gws)
    counts, offsets, hws = moe_expert_histogram_scan(ids, E, expert_map, ws=b.get("hist_ws"),
                                                     counts=b.get("counts"), offsets=b.get("offsets"))
    x_perm, perm_src, dest = moe_permute(x, ids, expert_map, hws, x_perm=b.get("x_perm"),
                                         perm_src=b.get("perm_src"), dest=b.get("dest"), gather=not fuse_gather)
    if fuse_gather:
        y_perm, fws = moe_grouped_swiglu_ffn_gather(x, perm_src, k, w_gate, w_up, w_down, offsets,
                                                    ws=b.get("ffn_ws"), y_perm=b.get("y_perm"))
    else:
        y_perm, fws = moe_grouped_swiglu_ffn(x_perm, w_gate, w_up, w_down, offsets, ws=b.get("ffn_ws"),
                                             y_perm=b.get("y_perm"))
    out = moe_unpermute_combine(y_perm, wts, dest, T, out=b.get("out"))
    if bufs is not None:
        bufs.update(ids=ids, weights=wts, gate_ws=gws, hist_ws=hws, counts=counts, offsets=offsets, perm_src=perm_src,
                    dest=dest, ffn_ws=fws, y_perm=y_perm, out=out)
        if x_perm is not None:
            bufs["x_perm"] = x_perm
    return dict(ids=ids, weights=wts, logits=lg, counts=counts, offsets=offsets, x_perm=x_perm,
                perm_src=perm_src, dest=dest, y_perm=y_perm, h=fws, out=out)


FFN_COUNTER_BYTES = 16384  # bf16 FFN workspace: counters first, then h


def ffn_hidden(ws, M_cap, I, dtype):
    """View of the expert hidden activations h [M_cap, I] held in an FFN workspace."""
    es = 2 if dtype == torch.bfloat16 else 4
    off = FFN_COUNTER_BYTES if dtype == torch.bfloat16 else 0
    return ws[off: off + M_cap * I * es].view(dtype).view(M_cap, I)


# ---------------------------------------------------------------------------
# Placement control path (latency model, greedy placement, drift, swaps)
# ---------------------------------------------------------------------------
def moe_fit_latency_model(loads, latencies):
    """Knots (n, t) of a monotone latency model from measured points (host)."""
    L = load_library()
    ld = np.ascontiguousarray(np.asarray(loads, dtype=np.int32))
    lt = np.ascontiguousarray(np.asarray(latencies, dtype=np.float32))
    if ld.shape != lt.shape or ld.ndim != 1:
        raise ValueError("loads and latencies must be 1-D of equal length")
    kn = np.zeros(len(ld), np.float64)
    kt = np.zeros(len(ld), np.float64)
    st = L.moe_fit_latency_model(ld.ctypes.data_as(_P), lt.ctypes.data_as(_P), len(ld), kn.ctypes.data_as(_P),
                                 kt.ctypes.data_as(_P))
    _check("moe_fit_latency_model", st)
    return kn, kt


def _models(knots_n, knots_t):
    if knots_n.dim() != 2 or knots_n.shape != knots_t.shape:
        raise ValueError("knots_n and knots_t must both be [G, nk]")
    return _dev(knots_n, "knots_n", torch.float64), _dev(knots_t, "knots_t", torch.float64), *knots_n.shape


def moe_place_greedy(w, knots_n, knots_t, cap=0, assign=None, loads=None, targets=None):
    """Latency-aware greedy placement of every layer. Returns (assign [L,E] int32,
    loads [L,G] fp64, targets [L,G] fp64)."""
    L = load_library()
    nl, E = w.shape
    kn, kt, G, nk = _models(knots_n, knots_t)
    assign = torch.empty((nl, E), dtype=torch.int32, device=w.device) if assign is None else assign
    loads = torch.empty((nl, G), dtype=torch.float64, device=w.device) if loads is None else loads
    targets = torch.empty((nl, G), dtype=torch.float64, device=w.device) if targets is None else targets
    st = L.moe_place_greedy(_dev(w, "w", torch.float64), nl, E, kn, kt, G, nk, cap,
                            _dev(assign, "assign", torch.int32), _dev(loads, "loads", torch.float64),
                            _dev(targets, "targets", torch.float64), _stream())
    _check("moe_place_greedy", st)
    return assign, loads, targets


def moe_place_incremental(w, knots_n, knots_t, assign, eps=0.03, max_swaps=1 << 16, n_swaps=None):
    """Swap-based placement update of every layer; `assign` is updated in place.
    Returns n_swaps [L] int32."""
    L = load_library()
    nl, E = w.shape
    kn, kt, G, nk = _models(knots_n, knots_t)
    n_swaps = torch.empty(nl, dtype=torch.int32, device=w.device) if n_swaps is None else n_swaps
    st = L.moe_place_incremental(_dev(w, "w", torch.float64), nl, E, kn, kt, G, nk, float(eps), int(max_swaps),
                                 _dev(assign, "assign", torch.int32), _dev(n_swaps, "n_swaps", torch.int32),
                                 _stream())
    _check("moe_place_incremental", st)
    return n_swaps


def moe_placement_cost(w, assign, knots_n, knots_t):
    """Per layer and GPU: loads n_g, f_g(n_g) and sum_{e in S_g} f_g(w_e).
    Returns (loads, lat, lat_grouped), each [L, G] fp64."""
    L = load_library()
    nl, E = w.shape
    kn, kt, G, nk = _models(knots_n, knots_t)
    out = [torch.empty((nl, G), dtype=torch.float64, device=w.device) for _ in range(3)]
    st = L.moe_placement_cost(_dev(w, "w", torch.float64), _dev(assign, "assign", torch.int32), nl, E, kn, kt, G, nk,
                              *[_dev(o, "out", torch.float64) for o in out], _stream())
    _check("moe_placement_cost", st)
    return tuple(out)


def moe_window_push(counts, ring, sums, slot):
    """sums += counts - ring[slot]; ring[slot] = counts (all on the GPU)."""
    L = load_library()
    window, nl, E = ring.shape
    if tuple(counts.shape) != (nl, E) or tuple(sums.shape) != (nl, E):
        raise ValueError("counts and sums must be [L, E] like ring[slot]")
    st = L.moe_window_push(_dev(counts, "counts", torch.int32), _dev(ring, "ring", torch.int32),
                           _dev(sums, "sums", torch.float64), nl, E, window, int(slot), _stream())
    _check("moe_window_push", st)


def moe_drift_distance(w_cur, w_ref, delta=0.05, d=None, trigger=None):
    """Cosine distance per layer and the drift trigger. Returns (d [L], trigger [1])."""
    L = load_library()
    nl, E = w_cur.shape
    if tuple(w_ref.shape) != (nl, E):
        raise ValueError("w_ref must match w_cur")
    d = torch.empty(nl, dtype=torch.float64, device=w_cur.device) if d is None else d
    trigger = torch.empty(1, dtype=torch.int32, device=w_cur.device) if trigger is None else trigger
    st = L.moe_drift_distance(_dev(w_cur, "w_cur", torch.float64), _dev(w_ref, "w_ref", torch.float64), nl, E,
                              float(delta), _dev(d, "d", torch.float64), _dev(trigger, "trigger", torch.int32),
                              _stream())
    _check("moe_drift_distance", st)
    return d, trigger


# ---------------------------------------------------------------------------
# MXFP8 expert FFN
# ---------------------------------------------------------------------------
class MxTensor:
    """An MXFP8 operand: E4M3 codes [.., R, K] uint8 and scale dwords
    [.., K/128, R] int32 (byte b of dword (k, r): the E8M0 code of elements
    [128 k + 32 b, +32) of row r). The codes may be a view with padded rows
    (row stride ld >= K bytes, matrices R * ld apart), which weight operands
    accept."""

    def __init__(self, codes, scales):
        if codes.dtype != torch.uint8 or scales.dtype != torch.int32:
            raise ValueError("MXFP8 codes are uint8 and scales int32")
        R, K = codes.shape[-2:]
        if tuple(scales.shape[-2:]) != (K // 128, R) or codes.shape[:-2] != scales.shape[:-2]:
            raise ValueError("scales must be [.., K/128, R] for codes [.., R, K]")
        ld = codes.stride(-2) if R > 1 and codes.numel() > 0 else K
        if codes.numel() > 0 and (codes.stride(-1) != 1 or ld < K or (codes.dim() == 3 and codes.shape[0] > 1
                                                                       and codes.stride(0) != R * ld)):
            raise ValueError("MXFP8 codes must be dense or rows padded to a common stride")
        self.codes, self.scales, self.ld = codes, scales, ld

    @property
    def shape(self):
        return tuple(self.codes.shape)


def moe_mx_quantize(x, out=None, row_count=None, ld=None):
    """MXFP8 quantisation of x [R, K] or [B, R, K] (bf16 or fp32) along K.
    row_count: optional device int32 tensor of one element (R-row x only):
    rows from it on are left as they are in `out`. ld: row stride in bytes
    of newly allocated codes (weights: ``weight_row_stride(K, 1)``)."""
    L = load_library()
    xb = x.unsqueeze(0) if x.dim() == 2 else x
    B, R, K = xb.shape
    if out is None:
        ld = K if ld is None else ld
        codes = torch.empty(tuple(x.shape[:-1]) + (ld,), dtype=torch.uint8, device=x.device)[..., :K]
        out = MxTensor(codes, torch.empty(tuple(x.shape[:-2]) + (K // 128, R), dtype=torch.int32,
                                          device=x.device))
    rc = ctypes.c_void_p(None)
    if row_count is not None:
        if row_count.numel() != 1 or row_count.dtype != torch.int32 or not row_count.is_cuda:
            raise ValueError("row_count must be one device int32")
        rc = ctypes.c_void_p(row_count.data_ptr())
    st = L.moe_mx_quantize(_dev(x, "x"), _dtype_code(x), B, R, K, out.ld, rc, _mx_codes(out.codes, "codes"),
                           _dev(out.scales, "scales", torch.int32), _stream())
    _check("moe_mx_quantize", st)
    return out


def _mx_codes(c, name):
    if not c.is_cuda:
        raise ValueError(f"{name} must be on the GPU (libmoe has no CPU path)")
    return ctypes.c_void_p(c.data_ptr())


def _mx_dev(t, name, shape, padded=False):
    """Pointers of an MXFP8 operand; only weight operands (padded=True) may
    have padded code rows."""
    if not isinstance(t, MxTensor):
        raise TypeError(f"{name} must be an MxTensor")
    if t.shape != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {t.shape}")
    if not padded and t.ld != t.shape[-1]:
        raise ValueError(f"{name} must have dense code rows")
    return _mx_codes(t.codes, name + ".codes"), _dev(t.scales, name + ".scales", torch.int32)


def moe_grouped_swiglu_mx(x, w_gate, w_up, offsets, h=None):
    """Gate/up half of the MXFP8 FFN: h = MXFP8(silu(x Wg^T) * (x Wu^T)) per local expert."""
    L = load_library()
    M_cap, H = x.shape
    E_local, I, _ = w_gate.shape
    if offsets.numel() != E_local + 1:
        raise ValueError("offsets must have E_local + 1 entries")
    dev = x.codes.device
    if h is None:
        h = MxTensor(torch.empty((M_cap, I), dtype=torch.uint8, device=dev),
                     torch.empty((I // 128, M_cap), dtype=torch.int32, device=dev))
    if w_up.ld != w_gate.ld:
        raise ValueError("w_gate and w_up must have the same row stride")
    st = L.moe_grouped_swiglu_mx(*_mx_dev(x, "x", (M_cap, H)), *_mx_dev(w_gate, "w_gate", (E_local, I, H), True),
                                 *_mx_dev(w_up, "w_up", (E_local, I, H), True),
                                 _dev(offsets, "offsets", torch.int32), E_local, H, I, w_gate.ld, M_cap,
                                 *_mx_dev(h, "h", (M_cap, I)), _stream())
    _check("moe_grouped_swiglu_mx", st)
    return h


def moe_grouped_gemm_mx(a, b, offsets, c=None):
    """Grouped MXFP8 GEMM: c[R] = bf16(a[R] b[l]^T) per local expert l."""
    L = load_library()
    M_cap, K = a.shape
    E_local, N, _ = b.shape
    if offsets.numel() != E_local + 1:
        raise ValueError("offsets must have E_local + 1 entries")
    if c is None:
        c = torch.empty((M_cap, N), dtype=torch.bfloat16, device=a.codes.device)
    st = L.moe_grouped_gemm_mx(*_mx_dev(a, "a", (M_cap, K)), *_mx_dev(b, "b", (E_local, N, K), True),
                               _dev(offsets, "offsets", torch.int32), E_local, N, K, b.ld, M_cap,
                               _dev(c, "c", torch.bfloat16), _stream())
    _check("moe_grouped_gemm_mx", st)
    return c


def ffn_mx_ws_bytes(E_local, H, I, M_cap):
    L = load_library()
    n = ctypes.c_size_t(0)
    st = L.moe_grouped_swiglu_ffn_mx(None, None, None, None, None, None, None, None, None, E_local, H, I, 0, 0,
                                     M_cap, None, None, ctypes.byref(n), None)
    _check("moe_grouped_swiglu_ffn_mx", st)
    return n.value


def moe_grouped_swiglu_ffn_mx(x, w_gate, w_up, w_down, offsets, ws=None, y_perm=None):
    """MXFP8 expert FFN. Returns (y_perm [M_cap, H] bf16, ws); ws holds h codes
    [M_cap, I] at byte FFN_COUNTER_BYTES and h scales [I/128, M_cap] after
    them (256-aligned)."""
    L = load_library()
    M_cap, H = x.shape
    E_local, I, _ = w_gate.shape
    if offsets.numel() != E_local + 1:
        raise ValueError("offsets must have E_local + 1 entries")
    dev = x.codes.device
    if ws is None:
        ws = torch.zeros(ffn_mx_ws_bytes(E_local, H, I, M_cap), dtype=torch.uint8, device=dev)  # counters start at zero
    if y_perm is None:
        y_perm = torch.empty((M_cap, H), dtype=torch.bfloat16, device=dev)
    n = ctypes.c_size_t(ws.numel())
    if w_up.ld != w_gate.ld:
        raise ValueError("w_gate and w_up must have the same row stride")
    st = L.moe_grouped_swiglu_ffn_mx(*_mx_dev(x, "x", (M_cap, H)),
                                     *_mx_dev(w_gate, "w_gate", (E_local, I, H), True),
                                     *_mx_dev(w_up, "w_up", (E_local, I, H), True),
                                     *_mx_dev(w_down, "w_down", (E_local, H, I), True),
                                     _dev(offsets, "offsets", torch.int32), E_local, H, I, w_gate.ld, w_down.ld,
                                     M_cap,
                                     _dev(y_perm, "y_perm", torch.bfloat16), _dev(ws, "ws", torch.uint8),
                                     ctypes.byref(n), _stream())
    _check("moe_grouped_swiglu_ffn_mx", st)
    return y_perm, ws


def moe_load_sweep_mx(x, w_gate, w_up, w_down, Ms, warmup=3, iters=10, y_scratch=None, keep_all=False):
    """Latency vs token load of the MXFP8 FFN on one expert. x: MxTensor [maxM, H];
    weights: MxTensors [n_rot, I, H] / [n_rot, H, I]. Returns (median_us [nM], all_us or None)."""
    L = load_library()
    n_rot, I, H = w_gate.shape
    Ms = np.ascontiguousarray(np.asarray(Ms, dtype=np.int32))
    nM = len(Ms)
    max_m = int(Ms.max())
    if x.shape != (max_m, H):
        raise ValueError(f"x must be [{max_m}, {H}] (rows for the largest M)")
    dev = x.codes.device
    n = ctypes.c_size_t(0)
    if w_up.ld != w_gate.ld:
        raise ValueError("w_gate and w_up must have the same row stride")
    args = (*_mx_dev(x, "x", (max_m, H)), *_mx_dev(w_gate, "w_gate", (n_rot, I, H), True),
            *_mx_dev(w_up, "w_up", (n_rot, I, H), True), *_mx_dev(w_down, "w_down", (n_rot, H, I), True), n_rot,
            H, I, w_gate.ld, w_down.ld, Ms.ctypes.data_as(ctypes.c_void_p), nM, warmup, iters)
    st = L.moe_load_sweep_mx(*args, None, None, ctypes.byref(n), None, None, _stream())
    _check("moe_load_sweep_mx", st)
    ws = torch.zeros(n.value, dtype=torch.uint8, device=dev)  # counters start at zero
    y = torch.empty((max_m, H), dtype=torch.bfloat16, device=dev) if y_scratch is None else y_scratch
    med = np.zeros(nM, np.float32)
    allv = np.zeros((nM, iters), np.float32) if keep_all else None
    st = L.moe_load_sweep_mx(*args, _dev(y, "y_scratch", torch.bfloat16), _dev(ws, "ws"), ctypes.byref(n),
                             med.ctypes.data_as(ctypes.c_void_p),
                             allv.ctypes.data_as(ctypes.c_void_p) if keep_all else None, _stream())
    _check("moe_load_sweep_mx", st)
    return med, allv
