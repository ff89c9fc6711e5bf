"""Python binding of libsaki (ctypes).  Argument marshalling only.

Each function has the name of the C entry point it calls (include/saki.h)
and does no arithmetic of its own: host functions take and return numpy
arrays, GPU functions take torch CUDA tensors (torch supplies device memory
and the current HIP stream) and enqueue the library's kernels on that
stream.  If the shared library is missing, every call raises: there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsaki.so")
_lib = None

F32, BF16, FP8 = 0, 1, 2
METHOD_OPT, METHOD_KEY_PCA, METHOD_SHARED, METHOD_SAP_MAP, METHOD_SAP_SVD = 0, 1, 2, 3, 4
_DTYPES = {"f32": F32, "bf16": BF16, "fp8": FP8}
_METHODS = {"opt": METHOD_OPT, "key_pca": METHOD_KEY_PCA, "shared": METHOD_SHARED,
            "sap_map": METHOD_SAP_MAP, "sap_svd": METHOD_SAP_SVD}


class SakiError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn} failed with status {status}: {saki_status_string(status)}")
        self.status = status


def lib():
    """Load libsaki.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing; build it with "
                           "`python -m paper_2608_03228_amd.build`")
    L = C.CDLL(_LIB_PATH)
    vp, ip, dp = C.c_void_p, C.c_int, C.c_double
    sz = C.c_size_t
    sig = {
        "saki_status_string": (C.c_char_p, [ip]),
        "saki_version": (ip, []),
        "saki_calibrate": (ip, [vp, vp, ip, ip, ip, ip, ip, ip, dp, vp, vp, vp, vp, vp, ip]),
        "saki_weight_svd_factors": (ip, [vp, ip, ip, ip, ip, ip, vp, vp]),
        "saki_sym_eig": (ip, [ip, vp, vp, vp]),
        "saki_index_bytes": (sz, [ip, ip, ip, ip, ip]),
        "saki_build_index": (ip, [vp, ip, ip, ip, ip, ip, ip, ip, vp, vp, ip, vp, sz, ip, ip, vp]),
        "saki_index_export": (ip, [vp, ip, ip, ip, ip, ip, vp, vp]),
        "saki_calibration_moments": (ip, [vp, vp, ip, ip, ip, ip, vp, vp, vp, vp]),
        "saki_calibrate_from_moments": (ip, [vp, vp, vp, ip, ip, ip, ip, ip, dp, vp, vp, vp, vp,
                                             vp, ip]),
        "saki_score_topk_workspace_bytes": (sz, [ip, ip, ip, ip, ip, ip, ip, ip]),
        "saki_score_topk": (ip, [vp, ip, ip, ip, ip, ip, ip, ip, ip, ip, vp, vp, ip, vp, vp, ip,
                                 vp, vp, vp, sz, vp]),
        "saki_score_topk_noalloc": (ip, [vp, ip, ip, ip, ip, ip, ip, ip, ip, ip, vp, vp, ip, vp,
                                         vp, ip, vp, vp, vp]),
        "saki_noalloc_scratch_bytes": (sz, []),
        "saki_recall_workspace_bytes": (sz, [ip, ip, ip, ip, ip, ip, ip]),
        "saki_recall": (ip, [vp, ip, vp, vp, ip, ip, ip, ip, ip, ip, ip, ip, vp, vp, vp, vp,
                             sz, vp]),
        "saki_attend": (ip, [vp, ip, vp, vp, ip, ip, ip, ip, ip, ip, ip, ip, ip, ip, vp, vp, ip,
                             vp, vp, vp, ip, C.c_float, vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def saki_status_string(status: int) -> str:
    return lib().saki_status_string(int(status)).decode()


def saki_version() -> int:
    return lib().saki_version()


def _check(fn, status):
    if status != 0:
        raise SakiError(fn, status)


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(C.c_void_p)


# ------------------------------------------------------------------ host calls

def saki_calibrate(q_cal, k_cal, r: int, method: str = "opt", floor_rel: float = 1e-6,
                   n_threads: int = 0, with_sigma: bool = True):
    """q_cal [H_q, T, d], k_cal [H_kv, T, d] (float32) -> dict of numpy arrays
    B_q, B_k [H_q, d, r] float32, mu [H_kv, d] float32, sigma [H_q, d] float64
    (None without with_sigma, which lets the library compute only the r
    largest singular values), n_clamped [H_q, 2] int32."""
    q, qp = _host(q_cal, np.float32)
    k, kp = _host(k_cal, np.float32)
    if q.ndim != 3 or k.ndim != 3 or q.shape[1:] != k.shape[1:]:
        raise ValueError("q_cal [H_q, T, d] and k_cal [H_kv, T, d] must agree in T and d")
    H_q, T, d = q.shape
    H_kv = k.shape[0]
    B_q = np.empty((H_q, d, r), np.float32)
    B_k = np.empty((H_q, d, r), np.float32)
    mu = np.empty((H_kv, d), np.float32)
    sigma = np.empty((H_q, d), np.float64) if with_sigma else None
    ncl = np.empty((H_q, 2), np.int32)
    st = lib().saki_calibrate(qp, kp, H_q, H_kv, T, d, int(r), _METHODS[method],
                              float(floor_rel), B_q.ctypes.data, B_k.ctypes.data,
                              mu.ctypes.data, sigma.ctypes.data if with_sigma else None,
                              ncl.ctypes.data, int(n_threads))
    _check("saki_calibrate", st)
    return {"B_q": B_q, "B_k": B_k, "mu": mu, "sigma": sigma, "n_clamped": ncl}


def saki_calibrate_from_moments(Sigma_q, Sigma_k, key_mean, r: int, method: str = "opt",
                                floor_rel: float = 1e-6, n_threads: int = 0,
                                with_sigma: bool = True, out=None):
    """Sigma_q [H_q, d, d], Sigma_k [H_kv, d, d], key_mean [H_kv, d] (float64,
    host) -> the same dict as saki_calibrate.  `out` may hold preallocated
    B_q, B_k, mu (and sigma, n_clamped) arrays."""
    sq, sqp = _host(Sigma_q, np.float64)
    sk, skp = _host(Sigma_k, np.float64)
    m, mp = _host(key_mean, np.float64)
    H_q, d = sq.shape[0], sq.shape[1]
    H_kv = sk.shape[0]
    o = out if out is not None else {}
    B_q = o.get("B_q", np.empty((H_q, d, r), np.float32))
    B_k = o.get("B_k", np.empty((H_q, d, r), np.float32))
    mu = o.get("mu", np.empty((H_kv, d), np.float32))
    sigma = o.get("sigma", np.empty((H_q, d), np.float64)) if with_sigma else None
    ncl = o.get("n_clamped", np.empty((H_q, 2), np.int32))
    st = lib().saki_calibrate_from_moments(
        sqp, skp, mp, H_q, H_kv, d, int(r), _METHODS[method], float(floor_rel),
        B_q.ctypes.data, B_k.ctypes.data, mu.ctypes.data,
        sigma.ctypes.data if with_sigma else None, ncl.ctypes.data, int(n_threads))
    _check("saki_calibrate_from_moments", st)
    return {"B_q": B_q, "B_k": B_k, "mu": mu, "sigma": sigma, "n_clamped": ncl}


def saki_weight_svd_factors(W_K, H_q: int, r: int):
    """W_K [H_kv, d, D] (float64) -> (B_q, B_k) [H_q, d, r] float32."""
    w, wp = _host(W_K, np.float64)
    H_kv, d, D = w.shape
    B_q = np.empty((H_q, d, r), np.float32)
    B_k = np.empty((H_q, d, r), np.float32)
    _check("saki_weight_svd_factors",
           lib().saki_weight_svd_factors(wp, int(H_q), H_kv, d, D, int(r), B_q.ctypes.data,
                                         B_k.ctypes.data))
    return B_q, B_k


def saki_sym_eig(A):
    """Symmetric A [n, n] (float64) -> (w ascending [n], V [n, n] columns)."""
    a, ap = _host(A, np.float64)
    n = a.shape[0]
    w = np.empty(n, np.float64)
    V = np.empty((n, n), np.float64)
    _check("saki_sym_eig", lib().saki_sym_eig(n, ap, w.ctypes.data, V.ctypes.data))
    return w, V


def saki_index_bytes(B: int, H_q: int, N_cap: int, r: int, sketch: str) -> int:
    return int(lib().saki_index_bytes(B, H_q, N_cap, r, _DTYPES[sketch]))


def saki_score_topk_workspace_bytes(B, H_q, Q, N_valid, r, k, sketch, index_heads=None) -> int:
    ih = H_q if index_heads is None else int(index_heads)
    return int(lib().saki_score_topk_workspace_bytes(B, H_q, ih, Q, N_valid, r, k,
                                                     _DTYPES[sketch]))


def saki_recall_workspace_bytes(B, H_q, H_kv, Q, N_valid, d, k) -> int:
    return int(lib().saki_recall_workspace_bytes(B, H_q, H_kv, Q, N_valid, d, k))


# ------------------------------------------------------------------ GPU calls

def _torch():
    import torch
    return torch


def _dev(t, dtypes, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _key_dtype(keys):
    torch = _torch()
    return BF16 if keys.dtype == torch.bfloat16 else F32


def saki_calibration_moments(q_cal, k_cal, Sigma_q=None, Sigma_k=None, key_mean=None,
                             stream=None):
    """q_cal [H_q, T, d], k_cal [H_kv, T, d] float32 CUDA -> (Sigma_q [H_q, d, d],
    Sigma_k [H_kv, d, d], key_mean [H_kv, d]) float64 CUDA tensors."""
    torch = _torch()
    qp = _dev(q_cal, (torch.float32,), "q_cal")
    kp = _dev(k_cal, (torch.float32,), "k_cal")
    H_q, T, d = q_cal.shape
    H_kv = k_cal.shape[0]
    dev = q_cal.device
    if Sigma_q is None:
        Sigma_q = torch.empty((H_q, d, d), dtype=torch.float64, device=dev)
    if Sigma_k is None:
        Sigma_k = torch.empty((H_kv, d, d), dtype=torch.float64, device=dev)
    if key_mean is None:
        key_mean = torch.empty((H_kv, d), dtype=torch.float64, device=dev)
    st = lib().saki_calibration_moments(
        qp, kp, H_q, H_kv, T, d, _dev(Sigma_q, (torch.float64,), "Sigma_q"),
        _dev(Sigma_k, (torch.float64,), "Sigma_k"), _dev(key_mean, (torch.float64,), "key_mean"),
        _stream(stream))
    _check("saki_calibration_moments", st)
    return Sigma_q, Sigma_k, key_mean


def saki_build_index(keys, B_k, mu, r: int, sketch: str, H_q: int, index=None,
                     n_begin: int = 0, n_count=None, stream=None):
    """keys [B, H_kv, N_cap, d] (float32 or bfloat16), B_k [H_q, d, r], mu
    [H_kv, d] (float32, CUDA).  Returns the index buffer (uint8 CUDA tensor),
    allocated if not given."""
    torch = _torch()
    kp = _dev(keys, (torch.float32, torch.bfloat16), "keys")
    B, H_kv, N_cap, d = keys.shape
    nbytes = saki_index_bytes(B, H_q, N_cap, r, sketch)
    if index is None:
        index = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=keys.device)
    n_count = N_cap - n_begin if n_count is None else n_count
    st = lib().saki_build_index(
        kp, _key_dtype(keys), B, int(H_q), H_kv, N_cap, d, int(r),
        _dev(B_k, (torch.float32,), "B_k"), _dev(mu, (torch.float32,), "mu"),
        _DTYPES[sketch], _dev(index, (torch.uint8,), "index"), index.numel(),
        int(n_begin), int(n_count), _stream(stream))
    _check("saki_build_index", st)
    return index


def saki_index_export(index, sketch: str, B: int, H_q: int, N_cap: int, r: int, stream=None):
    torch = _torch()
    out = torch.empty((B, H_q, N_cap, r), dtype=torch.float32, device=index.device)
    st = lib().saki_index_export(_dev(index, (torch.uint8,), "index"), _DTYPES[sketch], B, H_q,
                                 N_cap, r, out.data_ptr(), _stream(stream))
    _check("saki_index_export", st)
    return out


def saki_score_topk(index, sketch: str, q, B_q, mu, H_kv: int, N_cap: int, N_valid: int,
                    r: int, q_pos=None, k: int = 64, ws=None, top_idx=None, top_score=None,
                    with_scores: bool = True, stream=None, index_heads=None):
    """q [B, H_q, Q, d] float32 CUDA; q_pos [Q] int32 CUDA or None; index_heads
    = code sets per sequence in the index (H_q, the default, or H_kv for a
    GQA-shared index).  Returns (top_idx [B, H_q, Q, k] int32, top_score
    float32 or None)."""
    torch = _torch()
    qp = _dev(q, (torch.float32,), "q")
    B, H_q, Q, d = q.shape
    ih = H_q if index_heads is None else int(index_heads)
    need = saki_score_topk_workspace_bytes(B, H_q, Q, N_valid, r, k, sketch, ih)
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    if top_idx is None:
        top_idx = torch.empty((B, H_q, Q, k), dtype=torch.int32, device=q.device)
    if with_scores and top_score is None:
        top_score = torch.empty((B, H_q, Q, k), dtype=torch.float32, device=q.device)
    pos = _dev(q_pos, (torch.int32,), "q_pos") if q_pos is not None else None
    st = lib().saki_score_topk(
        _dev(index, (torch.uint8,), "index"), _DTYPES[sketch], B, H_q, int(H_kv), ih, int(N_cap),
        int(N_valid), d, int(r), qp, pos, Q, _dev(B_q, (torch.float32,), "B_q"),
        _dev(mu, (torch.float32,), "mu"), int(k), _dev(top_idx, (torch.int32,), "top_idx"),
        _dev(top_score, (torch.float32,), "top_score") if with_scores else None,
        _dev(ws, (torch.uint8,), "ws"), ws.numel(), _stream(stream))
    _check("saki_score_topk", st)
    return top_idx, (top_score if with_scores else None)


def saki_noalloc_scratch_bytes() -> int:
    return int(lib().saki_noalloc_scratch_bytes())


def saki_score_topk_noalloc(index, sketch: str, q, B_q, mu, H_kv: int, N_cap: int,
                            N_valid: int, r: int, top_idx, top_score=None, q_pos=None,
                            k: int = 64, stream=None, index_heads=None):
    """saki_score_topk without a workspace (the library's static scratch
    array): the caller passes the outputs top_idx [B, H_q, Q, k] int32 and
    top_score float32 (or None)."""
    torch = _torch()
    qp = _dev(q, (torch.float32,), "q")
    B, H_q, Q, d = q.shape
    ih = H_q if index_heads is None else int(index_heads)
    pos = _dev(q_pos, (torch.int32,), "q_pos") if q_pos is not None else None
    st = lib().saki_score_topk_noalloc(
        _dev(index, (torch.uint8,), "index"), _DTYPES[sketch], B, H_q, int(H_kv), ih, int(N_cap),
        int(N_valid), d, int(r), qp, pos, Q, _dev(B_q, (torch.float32,), "B_q"),
        _dev(mu, (torch.float32,), "mu"), int(k), _dev(top_idx, (torch.int32,), "top_idx"),
        _dev(top_score, (torch.float32,), "top_score") if top_score is not None else None,
        _stream(stream))
    _check("saki_score_topk_noalloc", st)
    return top_idx, top_score


def saki_recall(keys, q, approx_idx, N_valid: int, q_pos=None, k: int = 64, ws=None,
                hits=None, exact_idx=None, want_exact: bool = True, stream=None):
    """keys [B, H_kv, N_cap, d], q [B, H_q, Q, d], approx_idx [B, H_q, Q, k]
    (CUDA).  Returns (hits [B, H_q, Q] int32, exact_idx [B, H_q, Q, k] or None)."""
    torch = _torch()
    kp = _dev(keys, (torch.float32, torch.bfloat16), "keys")
    qp = _dev(q, (torch.float32,), "q")
    B, H_kv, N_cap, d = keys.shape
    _, H_q, Q, _ = q.shape
    need = saki_recall_workspace_bytes(B, H_q, H_kv, Q, N_valid, d, k)
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    if hits is None:
        hits = torch.empty((B, H_q, Q), dtype=torch.int32, device=q.device)
    if want_exact and exact_idx is None:
        exact_idx = torch.empty((B, H_q, Q, k), dtype=torch.int32, device=q.device)
    pos = _dev(q_pos, (torch.int32,), "q_pos") if q_pos is not None else None
    st = lib().saki_recall(
        kp, _key_dtype(keys), qp, pos, B, H_q, H_kv, N_cap, int(N_valid), Q, d, int(k),
        _dev(approx_idx, (torch.int32,), "approx_idx"), _dev(hits, (torch.int32,), "hits"),
        _dev(exact_idx, (torch.int32,), "exact_idx") if want_exact else None,
        _dev(ws, (torch.uint8,), "ws"), ws.numel(), _stream(stream))
    _check("saki_recall", st)
    return hits, (exact_idx if want_exact else None)


KEYS_EXACT, KEYS_RECONSTRUCTED = 0, 1
ROPE_THETA = 500000.0


def saki_attend(values, q, top_idx, N_valid: int, keys=None, index=None, sketch: str = "bf16",
                B_q=None, mu=None, r: int = 32, index_heads=None, q_pos=None,
                rope_theta: float = ROPE_THETA, out=None, stream=None):
    """Attention of every (sequence, head, query) row over its listed keys in
    RoPE space.  values [B, H_kv, N_cap, d] f32, q [B, H_q, Q, d] f32,
    top_idx [B, H_q, Q, k] int32 (CUDA).  Keys come from `keys` (exact) or,
    when `keys` is None, are reconstructed as mu + B_q c from `index`.
    Returns out [B, H_q, Q, d] float32."""
    torch = _torch()
    vp_ = _dev(values, (torch.float32,), "values")
    qp = _dev(q, (torch.float32,), "q")
    B, H_kv, N_cap, d = values.shape
    _, H_q, Q, _ = q.shape
    k = top_idx.shape[-1]
    if out is None:
        out = torch.empty((B, H_q, Q, d), dtype=torch.float32, device=q.device)
    recon = keys is None
    pos = _dev(q_pos, (torch.int32,), "q_pos") if q_pos is not None else None
    st = lib().saki_attend(
        None if recon else _dev(keys, (torch.float32, torch.bfloat16), "keys"),
        F32 if recon else _key_dtype(keys), vp_,
        _dev(index, (torch.uint8,), "index") if recon else None, _DTYPES[sketch],
        KEYS_RECONSTRUCTED if recon else KEYS_EXACT, B, H_q, H_kv,
        int(index_heads if index_heads is not None else H_q), N_cap, int(N_valid), d, int(r), qp,
        pos, Q, _dev(B_q, (torch.float32,), "B_q") if recon else None,
        _dev(mu, (torch.float32,), "mu") if recon else None,
        _dev(top_idx, (torch.int32,), "top_idx"), int(k), float(rope_theta),
        _dev(out, (torch.float32,), "out"), _stream(stream))
    _check("saki_attend", st)
    return out
