"""Codebook file format, oracle-side reader and writer.

Test infrastructure only.  The file persists the two shared offline objects of
the codec (Sec. 3: the rotation Pi and the codebook C); the layout is this
project's own definition, all little-endian:

    offset  size      field
    0       8         magic  b"FIBQCB01"
    8       4 x u32   d, k, N, reserved (0)
    24      2 x u64   rotation seed, codebook seed
    40      N*k f32   C, row-major (codeword n at n*k)
    ..      d*d f32   Pi, row-major (y_i = sum_j Pi_ij x_j)
    ..      u64       FNV-1a 64-bit hash of every preceding byte
"""
import struct

import numpy as np

MAGIC = b"FIBQCB01"
FNV_OFFSET = 0xCBF29CE484222325
FNV_PRIME = 0x100000001B3


def fnv1a64(data):
    h = FNV_OFFSET
    for byte in data:
        h ^= byte
        h = (h * FNV_PRIME) & 0xFFFFFFFFFFFFFFFF
    return h


def dumps(d, k, N, C, Pi, seeds=(0, 0)):
    body = MAGIC + struct.pack("<4I2Q", d, k, N, 0, seeds[0], seeds[1])
    body += np.ascontiguousarray(C, dtype="<f4").tobytes()
    body += np.ascontiguousarray(Pi, dtype="<f4").tobytes()
    return body + struct.pack("<Q", fnv1a64(body))


def loads(blob):
    """-> dict(d, k, N, C float32 [N,k], Pi float32 [d,d], seeds); raises ValueError."""
    if len(blob) < 48 or blob[:8] != MAGIC:
        raise ValueError("not a codebook file")
    d, k, N, _, s0, s1 = struct.unpack_from("<4I2Q", blob, 8)
    need = 40 + 4 * (N * k + d * d) + 8
    if len(blob) != need:
        raise ValueError("codebook file has the wrong size")
    (h,) = struct.unpack_from("<Q", blob, need - 8)
    if h != fnv1a64(blob[:need - 8]):
        raise ValueError("codebook file checksum mismatch")
    C = np.frombuffer(blob, dtype="<f4", count=N * k, offset=40).reshape(N, k)
    Pi = np.frombuffer(blob, dtype="<f4", count=d * d, offset=40 + 4 * N * k).reshape(d, d)
    return dict(d=d, k=k, N=N, C=C.copy(), Pi=Pi.copy(), seeds=(s0, s1))
