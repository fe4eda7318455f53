"""fibq_attn_decode_noalloc (the attention entry point that allocates nothing)
against fibq_attn_decode with a caller workspace, through the C ABI.

Two calls in a row on the library's static scratch, the second with a
smaller problem (fewer groups, fewer tokens, a ragged tail), each compared
with the workspace entry point on the same inputs to the attention
tolerance: 2e-3 relative l2 per (group, head) and 2e-3 of the head's largest
entry elementwise.  The shapes cover the 4-bit (k = 8, N = 16) and 6-bit
(k = 8, N = 64) kernels and the k = 4 kernel; a problem larger than the
static scratch is refused before anything runs.
"""
import ctypes

import numpy as np
import pytest
import torch

import paper_2605_11478_amd as fq
from oracle import codec as occ

from _fixtures import oracle_rotation, quick_codebook
import gpu_helpers as gh

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _problem(device, d, k, N, G, n_g, T, seed):
    rng = np.random.default_rng(seed)
    P = occ.payload_bytes(d, k, N)
    kp = occ.pack(rng.integers(0, N, (n_g * T, d // k)), N).reshape(n_g, T, P)
    vp = occ.pack(rng.integers(0, N, (n_g * T, d // k)), N).reshape(n_g, T, P)
    kh = (np.abs(rng.standard_normal((n_g, T))) * 20).astype(np.float16)
    vh = (np.abs(rng.standard_normal((n_g, T))) * 20).astype(np.float16)
    q = rng.standard_normal((n_g, G, d)).astype(np.float32)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    return (t(q).to(torch.bfloat16), t(kp), t(occ.fp16_bits(kh).view(np.int16)), t(vp),
            t(occ.fp16_bits(vh).view(np.int16)))


def _abi_noalloc(q, kp, kn, vp, vn, T, k, N, Rd, Cd, out):
    n_g, G, d = q.shape
    return fq.lib().fibq_attn_decode_noalloc(
        q.data_ptr(), fq.BF16, kp.data_ptr(), kn.data_ptr(), vp.data_ptr(), vn.data_ptr(), n_g, G,
        T, kp.shape[1], d, k, fq.rate(k, N), N, Rd.data_ptr(), Cd.data_ptr(), 0.0, out.data_ptr(),
        torch.cuda.current_stream().cuda_stream)


def _abi_workspace(q, kp, kn, vp, vn, T, k, N, Rd, Cd, out):
    n_g, G, d = q.shape
    need = fq.attn_workspace_bytes(n_g, G, T, d, k, N)
    ws = torch.zeros((max(need, 1),), dtype=torch.uint8, device=q.device)
    rc = fq.lib().fibq_attn_decode(
        q.data_ptr(), fq.BF16, kp.data_ptr(), kn.data_ptr(), vp.data_ptr(), vn.data_ptr(), n_g, G,
        T, kp.shape[1], d, k, fq.rate(k, N), N, Rd.data_ptr(), Cd.data_ptr(), 0.0, out.data_ptr(),
        ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return rc


@pytest.mark.parametrize("d,k,N,G,big,small", [
    (64, 8, 16, 8, (24, 8192), (5, 1000)),
    (64, 8, 64, 8, (16, 4096), (3, 777)),
    (64, 4, 256, 8, (12, 2048), (4, 333)),
])
def test_noalloc_matches_workspace_entry(d, k, N, G, big, small, device):
    R, C = oracle_rotation(d), quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    for call, (n_g, T) in enumerate((big, small)):
        _say(f"[noalloc] d={d} k={k} N={N} G={G} call {call}: {n_g} groups x {T} tokens")
        args = _problem(device, d, k, N, G, n_g, T, seed=17 * call + N)
        out = torch.full((n_g, G, d), float("nan"), dtype=torch.float32, device=device)
        rc = _abi_noalloc(*args, T, k, N, Rd, Cd, out)
        assert rc == fq.FIBQ_OK, fq.strerror(rc)
        torch.cuda.synchronize()
        ref = torch.empty_like(out)
        assert _abi_workspace(*args, T, k, N, Rd, Cd, ref) == fq.FIBQ_OK
        o, r = out.cpu().numpy(), ref.cpu().numpy()
        assert np.isfinite(o).all()
        rel = gh.check_attention(o, r.astype(np.float64))
        _say(f"  max rel l2 against the workspace entry point: {rel:.2e}")


def test_noalloc_refuses_a_problem_beyond_the_scratch(device):
    """A problem whose workspace exceeds the static scratch is refused with
    FIBQ_EWORKSPACE and the output is left untouched."""
    d, k, N, G = 64, 2, 64, 8
    n_g, T = 16384, 64
    need = fq.attn_workspace_bytes(n_g, G, T, d, k, N)
    assert need > fq.ATTN_SCRATCH_BYTES
    R, C = oracle_rotation(d), quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    P = occ.payload_bytes(d, k, N)
    q = torch.zeros((n_g, G, d), dtype=torch.bfloat16, device=device)
    pay = torch.zeros((n_g, T, P), dtype=torch.uint8, device=device)
    nrm = torch.zeros((n_g, T), dtype=torch.int16, device=device)
    args = (q, pay, nrm, pay, nrm)
    out = torch.full((n_g, G, d), 7.0, dtype=torch.float32, device=device)
    _say(f"[noalloc] refusal: {need} bytes needed")
    assert _abi_noalloc(*args, T, k, N, Rd, Cd, out) == fq.FIBQ_EWORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    with pytest.raises(ValueError, match="static scratch"):
        fq.attn_decode_noalloc(*args, T, k, N, Rd, Cd, out=out)
