"""FibQuant random-access KV-cache codec on MI355X (gfx950).

Thin ctypes binding over ``libfibq.so`` (declared in ``include/fibq.h``):
argument marshalling only.  Every step of the codec runs in the library's HIP
kernels; there is no CPU fallback, and a missing library raises.

Tensors passed to device functions must be CUDA (HIP) tensors, contiguous,
on the current device; work is enqueued on torch's current stream.
"""
import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfibq.so")

FIBQ_OK = 0
FIBQ_EINVAL = -1
FIBQ_EUNSUPPORTED = -2
FIBQ_EHIP = -3
FIBQ_EIO = -4
FIBQ_EWORKSPACE = -5
F32, F16, BF16 = 0, 1, 2

_lib = None


class FibqError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} (status {status})")


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2605_11478_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        c_i, c_i64, c_u64, c_d, c_f, c_p = (ctypes.c_int, ctypes.c_int64, ctypes.c_uint64,
                                            ctypes.c_double, ctypes.c_float, ctypes.c_void_p)
        sig = {
            "fibq_strerror": (ctypes.c_char_p, [c_i]),
            "fibq_version": (c_i, []),
            "fibq_payload_bytes": (c_i, [c_i, c_i, c_i]),
            "fibq_supported": (c_i, [c_i, c_i, c_i]),
            "fibq_build_rotation": (c_i, [c_i, c_u64, c_p]),
            "fibq_build_codebook": (c_i, [c_i, c_i, c_d, c_i, c_u64, c_i64, c_i, c_i, c_i, c_p,
                                          c_p]),
            "fibq_build_codebook_init": (c_i, [c_i, c_i, c_d, c_i, c_u64, c_i64, c_i, c_i, c_i,
                                               c_i, c_i, c_p, c_p, c_p, c_p]),
            "fibq_encode_radius_first": (c_i, [c_p, c_i, c_i64, c_i64, c_i, c_i, c_d, c_i, c_i,
                                               c_p, c_p, c_p, c_p, c_p]),
            "fibq_build_parent_lists": (c_i, [c_p, c_i, c_i, c_i, c_i, c_i, c_p, c_p, c_p]),
            "fibq_encode_list": (c_i, [c_p, c_i, c_i64, c_i64, c_i, c_i, c_d, c_i, c_i, c_i, c_i,
                                       c_p, c_p, c_p, c_p, c_p, c_p, c_p, c_p]),
            "fibq_save_codebook": (c_i, [ctypes.c_char_p, c_i, c_i, c_i, c_p, c_p, c_u64, c_u64]),
            "fibq_load_codebook": (c_i, [ctypes.c_char_p, c_p, c_p, c_p, c_p, c_p, c_p]),
            "fibq_encode": (c_i, [c_p, c_i, c_i64, c_i64, c_i, c_i, c_d, c_i, c_p, c_p, c_p, c_p,
                                  c_p]),
            "fibq_decode": (c_i, [c_p, c_p, c_p, c_i64, c_i64, c_i, c_i, c_d, c_i, c_p, c_p, c_p,
                                  c_p]),
            "fibq_attn_workspace_bytes": (ctypes.c_size_t, [c_i64, c_i, c_i64, c_i, c_i, c_i]),
            "fibq_attn_decode": (c_i, [c_p, c_i, c_p, c_p, c_p, c_p, c_i64, c_i, c_i64, c_i64,
                                       c_i, c_i, c_d, c_i, c_p, c_p, c_f, c_p, c_p,
                                       ctypes.c_size_t, c_p]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def strerror(status):
    return lib().fibq_strerror(status).decode()


def _check(status, where):
    if status != FIBQ_OK:
        raise FibqError(status, where)


def rate(k, N):
    """b = log2(N) / k bits per coordinate (Sec. 3.1)."""
    return math.log2(N) / k


def payload_bytes(d, k, N):
    P = lib().fibq_payload_bytes(d, k, N)
    if P < 0:
        raise FibqError(P, "fibq_payload_bytes")
    return P


# ----------------------------------------------------------------- host ----
def build_rotation(d, seed):
    R = np.empty((d, d), dtype=np.float32)
    _check(lib().fibq_build_rotation(d, seed, R.ctypes.data), "fibq_build_rotation")
    return R


FIBQ_INIT = {"beta": 0, "shell": 1, "multishell": 2}


def build_codebook(d, k, N, seed, M=0, restarts=4, iters=25, n_threads=0, init="beta",
                   return_shells=False, shells=0, metric=None):
    """(C, train_mse), plus the starting codebook's shell count if return_shells.
    init: "beta" (Eq. radii_main), "shell" (App. D) or "multishell" (App. E;
    ``shells`` > 0 fixes S, else every factor pair is tried).  ``metric``: a
    k x k symmetric positive definite matrix for the Mahalanobis objective."""
    C = np.empty((N, k), dtype=np.float32)
    mse = ctypes.c_double(0.0)
    n_shells = ctypes.c_int(0)
    Mt = None if metric is None else np.ascontiguousarray(metric, dtype=np.float64)
    if Mt is not None and Mt.shape != (k, k):
        raise ValueError("metric must be k x k")
    if init == "beta" and not return_shells and not shells and Mt is None:
        _check(lib().fibq_build_codebook(d, k, rate(k, N), N, seed, M, restarts, iters, n_threads,
                                         C.ctypes.data, ctypes.addressof(mse)),
               "fibq_build_codebook")
    else:
        _check(lib().fibq_build_codebook_init(d, k, rate(k, N), N, seed, M, restarts, iters,
                                              n_threads, FIBQ_INIT.get(init, -1), shells,
                                              None if Mt is None else Mt.ctypes.data,
                                              C.ctypes.data,
                                              ctypes.addressof(mse), ctypes.addressof(n_shells)),
               "fibq_build_codebook_init")
    if return_shells:
        return C, mse.value, n_shells.value
    return C, mse.value


def save_codebook(path, C, R, rotation_seed=0, codebook_seed=0):
    C = np.ascontiguousarray(C, dtype=np.float32)
    R = np.ascontiguousarray(R, dtype=np.float32)
    N, k = C.shape
    d = R.shape[0]
    _check(lib().fibq_save_codebook(os.fsencode(path), d, k, N, C.ctypes.data, R.ctypes.data,
                                    rotation_seed, codebook_seed), "fibq_save_codebook")


def load_codebook(path):
    d, k, N = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    seeds = (ctypes.c_uint64 * 2)()
    L = lib()
    _check(L.fibq_load_codebook(os.fsencode(path), ctypes.addressof(d), ctypes.addressof(k),
                                ctypes.addressof(N), None, None, ctypes.addressof(seeds)),
           "fibq_load_codebook")
    C = np.empty((N.value, k.value), dtype=np.float32)
    R = np.empty((d.value, d.value), dtype=np.float32)
    _check(L.fibq_load_codebook(os.fsencode(path), ctypes.addressof(d), ctypes.addressof(k),
                                ctypes.addressof(N), C.ctypes.data, R.ctypes.data,
                                ctypes.addressof(seeds)), "fibq_load_codebook")
    return C, R, (seeds[0], seeds[1])


# --------------------------------------------------------------- device ----
def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    return {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}[t.dtype]


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    return t.data_ptr()


def _stream():
    return _torch().cuda.current_stream().cuda_stream


def encode(x, k, N, R, C, payload=None, norms=None):
    """x [n, d] (rows may be strided) -> (payload uint8 [n, P], norm bits int16 [n])."""
    torch = _torch()
    n, d = x.shape
    if x.stride(1) != 1:
        raise ValueError("x rows must be contiguous")
    P = payload_bytes(d, k, N)
    if payload is None:
        payload = torch.empty((n, P), dtype=torch.uint8, device=x.device)
    if norms is None:
        norms = torch.empty((n,), dtype=torch.int16, device=x.device)
    st = lib().fibq_encode(_dev(x, "x"), _dtype_code(x), n, x.stride(0), d, k, rate(k, N), N,
                           _dev(R, "R"), _dev(C, "C"), _dev(payload, "payload"),
                           _dev(norms, "norms"), _stream())
    _check(st, "fibq_encode")
    return payload, norms


def encode_radius_first(x, k, N, L, R, C, payload=None, norms=None):
    """Radius-first encoder over L shells (App. F Stage 1); as ``encode``."""
    torch = _torch()
    n, d = x.shape
    if x.stride(1) != 1:
        raise ValueError("x rows must be contiguous")
    P = payload_bytes(d, k, N)
    if payload is None:
        payload = torch.empty((n, P), dtype=torch.uint8, device=x.device)
    if norms is None:
        norms = torch.empty((n,), dtype=torch.int16, device=x.device)
    st = lib().fibq_encode_radius_first(_dev(x, "x"), _dtype_code(x), n, x.stride(0), d, k,
                                        rate(k, N), N, L, _dev(R, "R"), _dev(C, "C"),
                                        _dev(payload, "payload"), _dev(norms, "norms"),
                                        _stream())
    _check(st, "fibq_encode_radius_first")
    return payload, norms


def build_parent_lists(C, L, K, rounds=10):
    """Stage 2 tables (App. F) of a shell-major host codebook C [N, k]:
    (mu float64 [L, K, k], offsets int32 [L, K + 1], members int32 [N])."""
    C = np.ascontiguousarray(C, dtype=np.float32)
    N, k = C.shape
    mu = np.empty((L, K, k), dtype=np.float64)
    off = np.empty((L, K + 1), dtype=np.int32)
    mem = np.empty(N, dtype=np.int32)
    _check(lib().fibq_build_parent_lists(C.ctypes.data, N, k, L, K, rounds, mu.ctypes.data,
                                         off.ctypes.data, mem.ctypes.data),
           "fibq_build_parent_lists")
    return mu, off, mem


def encode_list(x, k, N, L, K, T, mu, offsets, members, R, C, payload=None, norms=None):
    """List-decoding encoder (App. F Stages 1 + 2); tables as device tensors."""
    torch = _torch()
    n, d = x.shape
    for t, name, dt, shape in ((mu, "mu", torch.float64, (L, K, k)),
                               (offsets, "offsets", torch.int32, (L, K + 1)),
                               (members, "members", torch.int32, (N,))):
        if t.dtype != dt or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {dt} tensor of shape {shape}")
    if x.stride(1) != 1:
        raise ValueError("x rows must be contiguous")
    P = payload_bytes(d, k, N)
    if payload is None:
        payload = torch.empty((n, P), dtype=torch.uint8, device=x.device)
    if norms is None:
        norms = torch.empty((n,), dtype=torch.int16, device=x.device)
    st = lib().fibq_encode_list(_dev(x, "x"), _dtype_code(x), n, x.stride(0), d, k, rate(k, N),
                                N, L, K, T, _dev(mu, "mu"), _dev(offsets, "offsets"),
                                _dev(members, "members"), _dev(R, "R"), _dev(C, "C"),
                                _dev(payload, "payload"), _dev(norms, "norms"), _stream())
    _check(st, "fibq_encode_list")
    return payload, norms


def decode(payload, norms, d, k, N, R, C, token_ids=None, out=None):
    """-> x_hat float32 [n, d]; rows token_ids (int64, device) or all rows."""
    torch = _torch()
    n_cache = payload.shape[0]
    n = n_cache if token_ids is None else token_ids.shape[0]
    if out is None:
        out = torch.empty((n, d), dtype=torch.float32, device=payload.device)
    ids = 0 if token_ids is None else _dev(token_ids, "token_ids")
    st = lib().fibq_decode(_dev(payload, "payload"), _dev(norms, "norms"), ids or None, n, n_cache,
                           d, k, rate(k, N), N, _dev(R, "R"), _dev(C, "C"), _dev(out, "out"),
                           _stream())
    _check(st, "fibq_decode")
    return out


def attn_workspace_bytes(n_groups, G, T, d, k, N):
    return lib().fibq_attn_workspace_bytes(n_groups, G, T, d, k, N)


def attn_decode(q, k_payload, k_norms, v_payload, v_norms, T, k, N, R, C, scale=0.0,
                workspace=None, out=None):
    """q [n_groups, G, d]; payloads [n_groups, T_stride, P]; norms [n_groups, T_stride].

    -> out float32 [n_groups, G, d].
    """
    torch = _torch()
    n_groups, G, d = q.shape
    T_stride = k_payload.shape[1]
    need = attn_workspace_bytes(n_groups, G, T, d, k, N)
    if workspace is None:
        workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty((n_groups, G, d), dtype=torch.float32, device=q.device)
    st = lib().fibq_attn_decode(_dev(q, "q"), _dtype_code(q), _dev(k_payload, "k_payload"),
                                _dev(k_norms, "k_norms"), _dev(v_payload, "v_payload"),
                                _dev(v_norms, "v_norms"), n_groups, G, T, T_stride, d, k,
                                rate(k, N), N, _dev(R, "R"), _dev(C, "C"), scale,
                                _dev(out, "out"), _dev(workspace, "workspace"),
                                workspace.numel(), _stream())
    _check(st, "fibq_attn_decode")
    return out
