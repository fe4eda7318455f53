"""The Python binding rejects bad tensors before any device entry point runs.

CPU only.  The library handle is wrapped so that the host-side queries
(payload size, workspace size, error text) still answer while any device
entry point fails the test: each bad argument must raise in the binding,
since the kernels index by the shapes they are given and a wrong dtype,
shape or stride would read or write outside the caller's allocations.
"""
import pytest
import torch

import paper_2605_11478_amd as fq

HOST_QUERIES = {"fibq_payload_bytes", "fibq_attn_workspace_bytes", "fibq_strerror"}


class _NoLaunch:
    def __init__(self, real):
        self._real = real

    def __getattr__(self, name):
        if name in HOST_QUERIES:
            return getattr(self._real, name)
        raise AssertionError(f"{name} was called: the binding let a bad argument through")


@pytest.fixture
def nolaunch(monkeypatch):
    real = fq.lib()
    monkeypatch.setattr(fq, "_lib", _NoLaunch(real))
    return real


d, k, N = 64, 8, 16
P = 4


def _rc():
    return torch.zeros((d, d), dtype=torch.float32), torch.zeros((N, k), dtype=torch.float32)


def _err(fn, match, exc=ValueError):
    with pytest.raises(exc, match=match):
        fn()


def test_encode_rejects_bad_tensors(nolaunch):
    R, C = _rc()
    x = torch.zeros((10, d), dtype=torch.bfloat16)
    _err(lambda: fq.encode(x.to(torch.int32), k, N, R, C), "x must have dtype")
    _err(lambda: fq.encode(x[:, ::2], k, N, R[:32, :32], C), "x rows must be contiguous")
    _err(lambda: fq.encode(x, k, N, R.double(), C), "R must have dtype")
    _err(lambda: fq.encode(x, k, N, R[:32], C), "R must have shape")
    _err(lambda: fq.encode(x, k, N, R, C[:8]), "C must have shape")
    _err(lambda: fq.encode(x, k, N, R.t(), C), "R must be contiguous")
    pay = torch.zeros((10, P), dtype=torch.uint8)
    nrm = torch.zeros((10,), dtype=torch.int16)
    _err(lambda: fq.encode(x, k, N, R, C, pay[:9], nrm), "payload must have shape")
    _err(lambda: fq.encode(x, k, N, R, C, pay.to(torch.int8), nrm), "payload must have dtype")
    _err(lambda: fq.encode(x, k, N, R, C, pay, nrm.to(torch.int32)), "norms must have dtype")
    _err(lambda: fq.encode(x, k, N, R, C, pay, nrm[:5]), "norms must have shape")
    # every argument right but on the host: the device check
    _err(lambda: fq.encode(x, k, N, R, C, pay, nrm), "must be a device tensor")


def test_decode_rejects_bad_tensors(nolaunch):
    R, C = _rc()
    pay = torch.zeros((20, P), dtype=torch.uint8)
    nrm = torch.zeros((20,), dtype=torch.int16)
    ids = torch.zeros((7,), dtype=torch.int64)
    _err(lambda: fq.decode(pay[:, :3], nrm, d, k, N, R, C), "payload must have shape")
    _err(lambda: fq.decode(pay, nrm[:19], d, k, N, R, C), "norms must have shape")
    _err(lambda: fq.decode(pay, nrm.float(), d, k, N, R, C), "norms must have dtype")
    _err(lambda: fq.decode(pay, nrm, d, k, N, R, C, token_ids=ids.int()), "token_ids must have dtype")
    _err(lambda: fq.decode(pay, nrm, d, k, N, R, C, token_ids=ids[::2]), "token_ids must be contiguous")
    _err(lambda: fq.decode(pay, nrm, d, k, N, R, C, token_ids=ids,
                           out=torch.zeros((6, d))), "out must have shape")
    _err(lambda: fq.decode(pay, nrm, d, k, N, R, C, out=torch.zeros((20, d), dtype=torch.float16)),
         "out must have dtype")
    _err(lambda: fq.decode(pay.t().contiguous().t(), nrm, d, k, N, R, C), "payload must be contiguous")
    _err(lambda: fq.decode(pay, nrm, d, k, N, R, C, token_ids=ids), "must be a device tensor")


def _attn_args(n_g=3, G=8, Ts=40):
    q = torch.zeros((n_g, G, d), dtype=torch.bfloat16)
    kp = torch.zeros((n_g, Ts, P), dtype=torch.uint8)
    kn = torch.zeros((n_g, Ts), dtype=torch.int16)
    return q, kp, kn, kp.clone(), kn.clone()


def test_attn_decode_rejects_bad_tensors(nolaunch):
    R, C = _rc()
    q, kp, kn, vp, vn = _attn_args()

    def call(**kw):
        a = dict(q=q, k_payload=kp, k_norms=kn, v_payload=vp, v_norms=vn, T=40, k=k, N=N, R=R,
                 C=C)
        a.update(kw)
        return lambda: fq.attn_decode(**a)

    _err(call(q=q.to(torch.int16)), "q must have dtype")
    _err(call(q=q[:, :, :32].contiguous()), "k_payload must have shape")  # d (so P) read from q
    _err(call(q=q[:2]), "k_payload must have shape")                    # group count
    _err(call(q=q.permute(1, 0, 2).contiguous().permute(1, 0, 2)), "q must be contiguous")
    _err(call(k_payload=kp[:, :, :3]), "k_payload must have shape")
    _err(call(k_payload=kp[:2]), "k_payload must have shape")
    _err(call(v_payload=vp[:, :39]), "v_payload must have shape")       # T_stride mismatch
    _err(call(v_payload=vp.to(torch.int8)), "v_payload must have dtype")
    _err(call(k_norms=kn[:, :39]), "k_norms must have shape")
    _err(call(v_norms=vn.to(torch.int32)), "v_norms must have dtype")
    _err(call(k_payload=kp[:, ::2]), "k_payload must be contiguous")   # strided view: 20 tokens
    _err(call(k_payload=kp[:, ::2], v_payload=vp[:, ::2], k_norms=kn[:, ::2], v_norms=vn[:, ::2],
              T=20), "k_payload must be contiguous")
    _err(call(T=41), "T = 41 must lie")
    _err(call(T=-1), "T = -1 must lie")
    _err(call(out=torch.zeros((3, 8, d), dtype=torch.float16)), "out must have dtype")
    _err(call(out=torch.zeros((3, 7, d))), "out must have shape")
    _err(call(workspace=torch.zeros((16,), dtype=torch.int32)), "workspace must have dtype")
    need = fq.attn_workspace_bytes(3, 8, 40, d, k, N)
    assert need > 16
    _err(call(workspace=torch.zeros((16,), dtype=torch.uint8)), f"{need} needed")
    _err(call(), "must be a device tensor")


def test_encode_list_rejects_bad_tables(nolaunch):
    R = torch.zeros((d, d), dtype=torch.float32)
    C = torch.zeros((256, 4), dtype=torch.float32)
    x = torch.zeros((10, d), dtype=torch.bfloat16)
    L, K, T = 16, 4, 2
    mu = torch.zeros((L, K, 4), dtype=torch.float64)
    off = torch.zeros((L, K + 1), dtype=torch.int32)
    mem = torch.zeros((256,), dtype=torch.int32)
    _err(lambda: fq.encode_list(x, 4, 256, L, K, T, mu.float(), off, mem, R, C), "mu must have dtype")
    _err(lambda: fq.encode_list(x, 4, 256, L, K, T, mu, off[:, :K], mem, R, C), "offsets must have shape")
    _err(lambda: fq.encode_list(x, 4, 256, L, K, T, mu, off, mem.long(), R, C), "members must have dtype")
    _err(lambda: fq.encode_list(x, 4, 256, L, K, T, mu, off, mem, R, C), "must be a device tensor")
