"""Random-access encoder / decoder (oracle side, float64).

Test infrastructure only.  Sec. 3.1 (Eq. encode):

* the norm header is nu = ||x||_2, stored as an fp16 value (IEEE
  round-to-nearest-even from the float64 norm);
* the rotated unit vector Pi x / nu is cut into d/k blocks of k consecutive
  coordinates, y^(m);
* block m stores i_m = argmin_j ||y^(m) - c_j||^2, by brute force over all N
  codewords, ties to the lowest index, 0-based;
* the decoder returns x_hat = nu_fp16 * Pi^T (c_{i_1}, ..., c_{i_{d/k}}).

Readings (the paper leaves these open): y is normalised by the unrounded norm
and only the stored header is fp16; an all-zero vector stores header 0 and
indices 0 and decodes to 0; the fixed-rate payload of a vector is
ceil(d * w / k / 8) bytes with w = log2 N, a little-endian bit stream in which
index m occupies bits [m w, (m + 1) w) (byte b holds bits 8b .. 8b+7, bit 0 the
least significant); unused trailing bits are zero.
"""
import math

import numpy as np


def index_bits(N):
    w = int(round(math.log2(N)))
    if 2 ** w != N:
        raise ValueError("N must be a power of two")
    return w


def payload_bytes(d, k, N):
    """Fixed payload size per vector: ceil((d/k) * log2(N) / 8) bytes (Sec. 3.1)."""
    return -(-(d // k) * index_bits(N) // 8)


def norms(x):
    """(nu float64, fp16 header) for each row of x (Sec. 3.1)."""
    x = np.asarray(x, dtype=np.float64)
    nu = np.sqrt((x * x).sum(axis=1))
    return nu, nu.astype(np.float16)


def rotate_normalise(x, Pi, nu):
    """y = Pi (x / nu) for each row; zero rows give y = 0."""
    x = np.asarray(x, dtype=np.float64)
    safe = np.where(nu > 0, nu, 1.0)
    return (x / safe[:, None]) @ np.asarray(Pi, dtype=np.float64).T


def block_distances(y, C, k):
    """D[v, m, j] = ||y^(m) - c_j||^2 for all vectors v, blocks m, codewords j."""
    C = np.asarray(C, dtype=np.float64)
    n, d = y.shape
    blocks = y.reshape(n, d // k, k)
    D = np.zeros((n, d // k, C.shape[0]))
    for i in range(k):
        D += (blocks[:, :, i:i + 1] - C[None, None, :, i]) ** 2
    return D


def encode(x, Pi, C, return_distances=False):
    """Encode rows of x -> (indices [n, d/k] int64, header fp16 [n]).

    With ``return_distances`` also returns D [n, d/k, N] (float64), used by
    the parity checker's near-tie window.
    """
    x = np.asarray(x, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    k = C.shape[1]
    nu, h = norms(x)
    y = rotate_normalise(x, Pi, nu)
    D = block_distances(y, C, k)
    idx = D.argmin(axis=2)
    zero = nu == 0
    idx[zero] = 0
    h[zero] = np.float16(0.0)
    if return_distances:
        return idx, h, D
    return idx, h


def decode(idx, h, Pi, C):
    """x_hat = fp16 header * Pi^T concat_m c_{i_m} for each vector (Sec. 3.1)."""
    C = np.asarray(C, dtype=np.float64)
    idx = np.asarray(idx)
    n = idx.shape[0]
    yhat = C[idx].reshape(n, -1)
    return np.asarray(h, dtype=np.float64)[:, None] * (yhat @ np.asarray(Pi, dtype=np.float64))


# ------------------------------------------------------------- bit packing ---
def pack(idx, N):
    """Indices [n, d/k] -> payload bytes [n, P] (little-endian bit stream)."""
    idx = np.asarray(idx, dtype=np.int64)
    w = index_bits(N)
    n, nb = idx.shape
    P = -(-nb * w // 8)
    out = np.zeros((n, P), dtype=np.uint8)
    for m in range(nb):
        for b in range(w):
            bit = (idx[:, m] >> b) & 1
            pos = m * w + b
            out[:, pos // 8] |= (bit << (pos % 8)).astype(np.uint8)
    return out


def unpack(payload, nblocks, N):
    """Payload bytes [n, P] -> indices [n, nblocks]."""
    payload = np.asarray(payload, dtype=np.uint8)
    w = index_bits(N)
    n = payload.shape[0]
    idx = np.zeros((n, nblocks), dtype=np.int64)
    for m in range(nblocks):
        for b in range(w):
            pos = m * w + b
            bit = (payload[:, pos // 8].astype(np.int64) >> (pos % 8)) & 1
            idx[:, m] |= bit << b
    return idx


def fp16_bits(h):
    return np.asarray(h, dtype=np.float16).view(np.uint16)


def from_fp16_bits(u):
    return np.asarray(u, dtype=np.uint16).view(np.float16)


def tie_ok(D, idx_ref, idx_got, rel=1e-6):
    """Near-tie rule of the parity checker: index j is accepted for a block iff
    j equals the oracle's index or D_j <= D_min * (1 + rel) on the oracle's
    float64 distances.  Returns a boolean array shaped like idx_ref."""
    D = np.asarray(D)
    idx_got = np.asarray(idx_got, dtype=np.int64)
    dmin = np.take_along_axis(D, np.asarray(idx_ref)[..., None], axis=-1)[..., 0]
    dgot = np.take_along_axis(D, idx_got[..., None], axis=-1)[..., 0]
    return (idx_got == idx_ref) | (dgot <= dmin * (1.0 + rel))
