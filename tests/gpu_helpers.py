"""Helpers for the GPU parity tests: oracle-side references and comparisons.

Reference values always come from ``oracle/`` applied to the same input bytes
that the device sees; nothing here reads a device result back into an oracle
input.
"""
import numpy as np
import torch

from oracle import attention as oat
from oracle import codec as occ

TIE_REL = 1e-6        # near-tie window on the oracle's float64 distances
RECON_TOL = 1e-5      # |x_hat_gpu - x_hat_ref| <= RECON_TOL * max(1, nu)
ATTN_TOL = 2e-3       # relative l2 per (group, head)


def host_f64(t):
    """Exact float64 copy of a device or host tensor (fp32/fp16/bf16)."""
    return t.detach().to("cpu").to(torch.float64).numpy()


def bits_u16(t):
    return t.detach().cpu().numpy().view(np.uint16)


def oracle_encode(x, R, C, chunk=256):
    """Oracle indices [n, d/k], fp16 headers, and per-block D rows needed for
    the tie rule, computed in chunks (D itself is n x d/k x N)."""
    n = x.shape[0]
    idx = np.empty((n, R.shape[0] // C.shape[1]), dtype=np.int64)
    h = np.empty(n, dtype=np.float16)
    Ds = []
    for s in range(0, n, chunk):
        i, hh, D = occ.encode(x[s:s + chunk], R.astype(np.float64), C.astype(np.float64),
                              return_distances=True)
        idx[s:s + chunk] = i
        h[s:s + chunk] = hh
        Ds.append(D)
    return idx, h, Ds


def check_indices(idx_ref, Ds, idx_gpu, chunk=256):
    """Tie rule: exact, or D_j <= D_min (1 + 1e-6).  Returns (n_exact, n_ties)."""
    n_exact = int((idx_ref == idx_gpu).sum())
    n_bad = 0
    worst = 0.0
    for c, D in enumerate(Ds):
        s = c * chunk
        ok = occ.tie_ok(D, idx_ref[s:s + D.shape[0]], idx_gpu[s:s + D.shape[0]], TIE_REL)
        n_bad += int((~ok).sum())
        if (~ok).any():
            dmin = np.take_along_axis(D, idx_ref[s:s + D.shape[0], :, None], -1)[..., 0]
            dgot = np.take_along_axis(D, idx_gpu[s:s + D.shape[0], :, None], -1)[..., 0]
            worst = max(worst, float(((dgot - dmin) / np.maximum(dmin, 1e-300))[~ok].max()))
    assert n_bad == 0, f"{n_bad} indices outside the tie window (worst rel gap {worst:.3e})"
    return n_exact, idx_ref.size - n_exact


def check_encode(x64, R, C, N, payload_gpu, norms_gpu):
    """Full encode parity for rows x64 (float64 exact copies of the inputs)."""
    d, k = R.shape[0], C.shape[1]
    idx_ref, h_ref, Ds = oracle_encode(x64, R, C)
    pay = payload_gpu.detach().cpu().numpy()
    idx_gpu = occ.unpack(pay, d // k, N)
    n_exact, n_ties = check_indices(idx_ref, Ds, idx_gpu)
    # byte layout: the device bytes are the oracle packing of the device indices
    assert np.array_equal(occ.pack(idx_gpu, N), pay)
    assert np.array_equal(bits_u16(norms_gpu), occ.fp16_bits(h_ref))
    return n_exact, n_ties, idx_ref, h_ref


def check_recon(xh_gpu, xh_ref, hdr):
    nu = np.abs(np.asarray(hdr, dtype=np.float64))
    tol = RECON_TOL * np.maximum(1.0, nu)[:, None]
    err = np.abs(xh_gpu.astype(np.float64) - xh_ref)
    assert np.all(err <= tol), f"max err/tol {float((err / tol).max()):.3f}"


def check_attention(o_gpu, o_ref):
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    num = np.linalg.norm(o_gpu - o_ref, axis=-1)
    den = np.linalg.norm(o_ref, axis=-1)
    rel = num / np.maximum(den, 1e-30)
    assert np.all(rel <= ATTN_TOL), f"max rel l2 {rel.max():.3e}"
    scale = np.abs(o_ref).max(axis=-1, keepdims=True)
    assert np.all(np.abs(o_gpu - o_ref) <= ATTN_TOL * np.maximum(scale, 1e-30))
    return float(rel.max())


def oracle_group_attention(q, kpay, knb, vpay, vnb, R, C, N, T):
    """Oracle attention for each group: q [n_g, G, d] float64; payload/norm bits
    [n_g, T_stride, ...] numpy; uses the first T tokens."""
    out = np.zeros(q.shape)
    for g in range(q.shape[0]):
        out[g] = oat.attention_from_payload(q[g], kpay[g, :T], knb[g, :T], vpay[g, :T],
                                            vnb[g, :T], R.astype(np.float64),
                                            C.astype(np.float64), N)
    return out
