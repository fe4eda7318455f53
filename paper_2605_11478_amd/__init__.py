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
            "fibq_attn_decode_noalloc": (c_i, [c_p, c_i, c_p, c_p, c_p, c_p, c_i64, c_i, c_i64,
                                               c_i64, c_i, c_i, c_d, c_i, c_p, c_p, c_f, c_p,
                                               c_p]),
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


def _norm_dtypes():
    torch = _torch()
    return tuple(dt for dt in (torch.int16, getattr(torch, "uint16", None)) if dt is not None)


def _want(t, name, dtypes, shape=None, contiguous=True):
    """Check one tensor argument before anything reaches the library: dtype (one
    of ``dtypes``), exact shape (None entries match any size) and density.
    The device is checked afterwards by ``_same_device``."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} must have dtype {' or '.join(str(d) for d in dtypes)}, "
                         f"got {t.dtype}")
    if shape is not None:
        if t.dim() != len(shape) or any(s is not None and t.shape[i] != s
                                        for i, s in enumerate(shape)):
            want = "[" + ", ".join("*" if s is None else str(s) for s in shape) + "]"
            raise ValueError(f"{name} must have shape {want}, got {list(t.shape)}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _same_device(**tensors):
    """Every tensor on one HIP device (the library reads them all from the
    current device's memory)."""
    devs = set()
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        devs.add(t.device)
    if len(devs) > 1:
        raise ValueError(f"tensors are on different devices: {sorted(map(str, devs))}")


def _check_rc(R, C, d, k, N):
    torch = _torch()
    _want(R, "R", (torch.float32,), (d, d))
    _want(C, "C", (torch.float32,), (N, k))


def _enc_outputs(x, n, P, payload, norms):
    torch = _torch()
    if payload is None:
        payload = torch.empty((n, P), dtype=torch.uint8, device=x.device)
    if norms is None:
        norms = torch.empty((n,), dtype=torch.int16, device=x.device)
    _want(payload, "payload", (torch.uint8,), (n, P))
    _want(norms, "norms", _norm_dtypes(), (n,))
    return payload, norms


def _check_x(x):
    torch = _torch()
    _want(x, "x", (torch.float32, torch.float16, torch.bfloat16), (None, None), contiguous=False)
    if x.stride(1) != 1 or (x.shape[0] > 1 and x.stride(0) < x.shape[1]):
        raise ValueError("x rows must be contiguous and must not overlap")


def encode(x, k, N, R, C, payload=None, norms=None):
    """x [n, d] (rows may be strided) -> (payload uint8 [n, P], norm bits int16 [n])."""
    _check_x(x)
    n, d = x.shape
    _check_rc(R, C, d, k, N)
    P = payload_bytes(d, k, N)
    payload, norms = _enc_outputs(x, n, P, payload, norms)
    _same_device(x=x, R=R, C=C, payload=payload, norms=norms)
    st = lib().fibq_encode(_dev(x, "x"), _dtype_code(x), n, x.stride(0), d, k, rate(k, N), N,
                           _dev(R, "R"), _dev(C, "C"), _dev(payload, "payload"),
                           _dev(norms, "norms"), _stream())
    _check(st, "fibq_encode")
    return payload, norms


def encode_radius_first(x, k, N, L, R, C, payload=None, norms=None):
    """Radius-first encoder over L shells (App. F Stage 1); as ``encode``."""
    _check_x(x)
    n, d = x.shape
    _check_rc(R, C, d, k, N)
    P = payload_bytes(d, k, N)
    payload, norms = _enc_outputs(x, n, P, payload, norms)
    _same_device(x=x, R=R, C=C, payload=payload, norms=norms)
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
    _check_x(x)
    n, d = x.shape
    _want(mu, "mu", (torch.float64,), (L, K, k))
    _want(offsets, "offsets", (torch.int32,), (L, K + 1))
    _want(members, "members", (torch.int32,), (N,))
    _check_rc(R, C, d, k, N)
    P = payload_bytes(d, k, N)
    payload, norms = _enc_outputs(x, n, P, payload, norms)
    _same_device(x=x, mu=mu, offsets=offsets, members=members, R=R, C=C, payload=payload,
                 norms=norms)
    st = lib().fibq_encode_list(_dev(x, "x"), _dtype_code(x), n, x.stride(0), d, k, rate(k, N),
                                N, L, K, T, _dev(mu, "mu"), _dev(offsets, "offsets"),
                                _dev(members, "members"), _dev(R, "R"), _dev(C, "C"),
                                _dev(payload, "payload"), _dev(norms, "norms"), _stream())
    _check(st, "fibq_encode_list")
    return payload, norms


def decode(payload, norms, d, k, N, R, C, token_ids=None, out=None):
    """-> x_hat float32 [n, d]; rows token_ids (int64, device) or all rows."""
    torch = _torch()
    P = payload_bytes(d, k, N)
    _want(payload, "payload", (torch.uint8,), (None, P))
    n_cache = payload.shape[0]
    _want(norms, "norms", _norm_dtypes(), (n_cache,))
    if token_ids is not None:
        _want(token_ids, "token_ids", (torch.int64,), (None,))
    n = n_cache if token_ids is None else token_ids.shape[0]
    _check_rc(R, C, d, k, N)
    if out is None:
        out = torch.empty((n, d), dtype=torch.float32, device=payload.device)
    _want(out, "out", (torch.float32,), (n, d))
    _same_device(payload=payload, norms=norms, token_ids=token_ids, R=R, C=C, out=out)
    ids = None if token_ids is None else _dev(token_ids, "token_ids")
    st = lib().fibq_decode(_dev(payload, "payload"), _dev(norms, "norms"), ids, n, n_cache,
                           d, k, rate(k, N), N, _dev(R, "R"), _dev(C, "C"), _dev(out, "out"),
                           _stream())
    _check(st, "fibq_decode")
    return out


def attn_workspace_bytes(n_groups, G, T, d, k, N):
    return lib().fibq_attn_workspace_bytes(n_groups, G, T, d, k, N)


def _check_attn(q, k_payload, k_norms, v_payload, v_norms, T, k, N, R, C, out):
    """Shapes of one attention call; returns (n_groups, G, d, T_stride, P, out)."""
    torch = _torch()
    _want(q, "q", (torch.float32, torch.float16, torch.bfloat16), (None, None, None))
    n_groups, G, d = q.shape
    P = payload_bytes(d, k, N)
    _want(k_payload, "k_payload", (torch.uint8,), (n_groups, None, P))
    T_stride = k_payload.shape[1]
    _want(v_payload, "v_payload", (torch.uint8,), (n_groups, T_stride, P))
    _want(k_norms, "k_norms", _norm_dtypes(), (n_groups, T_stride))
    _want(v_norms, "v_norms", _norm_dtypes(), (n_groups, T_stride))
    if not 0 <= T <= T_stride:
        raise ValueError(f"T = {T} must lie in [0, T_stride = {T_stride}]")
    _check_rc(R, C, d, k, N)
    if out is None:
        out = torch.empty((n_groups, G, d), dtype=torch.float32, device=q.device)
    _want(out, "out", (torch.float32,), (n_groups, G, d))
    return n_groups, G, d, T_stride, P, out


def attn_decode(q, k_payload, k_norms, v_payload, v_norms, T, k, N, R, C, scale=0.0,
                workspace=None, out=None):
    """q [n_groups, G, d]; payloads [n_groups, T_stride, P]; norms [n_groups, T_stride].

    -> out float32 [n_groups, G, d].  ``workspace`` (uint8, at least
    ``attn_workspace_bytes`` bytes) may be reused across calls that do not
    overlap in time; a fresh one is allocated (zero-filled) when omitted.
    """
    torch = _torch()
    n_groups, G, d, T_stride, P, out = _check_attn(q, k_payload, k_norms, v_payload, v_norms,
                                                   T, k, N, R, C, out)
    need = attn_workspace_bytes(n_groups, G, T, d, k, N)
    if workspace is None:
        workspace = torch.zeros((max(need, 1),), dtype=torch.uint8, device=q.device)
    _want(workspace, "workspace", (torch.uint8,), (None,))
    if workspace.numel() < need:
        raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
    _same_device(q=q, k_payload=k_payload, k_norms=k_norms, v_payload=v_payload,
                 v_norms=v_norms, R=R, C=C, out=out, workspace=workspace)
    st = lib().fibq_attn_decode(_dev(q, "q"), _dtype_code(q), _dev(k_payload, "k_payload"),
                                _dev(k_norms, "k_norms"), _dev(v_payload, "v_payload"),
                                _dev(v_norms, "v_norms"), n_groups, G, T, T_stride, d, k,
                                rate(k, N), N, _dev(R, "R"), _dev(C, "C"), scale,
                                _dev(out, "out"), _dev(workspace, "workspace"),
                                workspace.numel(), _stream())
    _check(st, "fibq_attn_decode")
    return out


# FIBQ_ATTN_SCRATCH_BYTES of include/fibq.h: the static workspace of
# attn_decode_noalloc on each GPU
ATTN_SCRATCH_BYTES = 64 << 20


def attn_decode_noalloc(q, k_payload, k_norms, v_payload, v_norms, T, k, N, R, C, scale=0.0,
                        out=None):
    """``attn_decode`` without a workspace: the library's static per-GPU
    scratch array is used instead (for callers that cannot allocate, e.g.
    under graph capture; pass ``out`` to allocate nothing at all).  Calls that
    overlap in time on one GPU race on that array."""
    n_groups, G, d, T_stride, P, out = _check_attn(q, k_payload, k_norms, v_payload, v_norms,
                                                   T, k, N, R, C, out)
    need = attn_workspace_bytes(n_groups, G, T, d, k, N)
    if need > ATTN_SCRATCH_BYTES:
        raise ValueError(f"this problem needs {need} bytes of workspace, more than the "
                         f"{ATTN_SCRATCH_BYTES} of the static scratch; use attn_decode")
    _same_device(q=q, k_payload=k_payload, k_norms=k_norms, v_payload=v_payload,
                 v_norms=v_norms, R=R, C=C, out=out)
    st = lib().fibq_attn_decode_noalloc(_dev(q, "q"), _dtype_code(q),
                                        _dev(k_payload, "k_payload"), _dev(k_norms, "k_norms"),
                                        _dev(v_payload, "v_payload"), _dev(v_norms, "v_norms"),
                                        n_groups, G, T, T_stride, d, k, rate(k, N), N,
                                        _dev(R, "R"), _dev(C, "C"), scale, _dev(out, "out"),
                                        _stream())
    _check(st, "fibq_attn_decode_noalloc")
    return out
