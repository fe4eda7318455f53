"""Naive single-query decode attention over the reconstructed cache (oracle side).

Test infrastructure only.  Eq. lattn: o = softmax(q K^T / sqrt(d)) V with K, V
replaced by the decoded cache K_hat, V_hat (Sec. 3.1 decoder).  Readings: no
mask (the single decoding query sees all T cached tokens); the scale defaults
to 1/sqrt(d); the softmax subtracts the row maximum before exponentiating;
with T = 0 the output is zero.
"""
import numpy as np

from . import codec


def attention(q, Khat, Vhat, scale=None):
    """q [G, d], Khat/Vhat [T, d] -> o [G, d] (float64)."""
    q = np.asarray(q, dtype=np.float64)
    Khat = np.asarray(Khat, dtype=np.float64)
    Vhat = np.asarray(Vhat, dtype=np.float64)
    G, d = q.shape
    if Khat.shape[0] == 0:
        return np.zeros((G, d))
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    s = (q @ Khat.T) * scale
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ Vhat


def attention_from_payload(q, k_payload, k_norm_bits, v_payload, v_norm_bits, Pi, C, N,
                           scale=None):
    """Decode one group's K and V (payload bytes + fp16 norm bits) and attend."""
    C = np.asarray(C, dtype=np.float64)
    d = np.asarray(Pi).shape[0]
    nb = d // C.shape[1]
    kh = codec.decode(codec.unpack(k_payload, nb, N), codec.from_fp16_bits(k_norm_bits), Pi, C)
    vh = codec.decode(codec.unpack(v_payload, nb, N), codec.from_fp16_bits(v_norm_bits), Pi, C)
    return attention(q, kh, vh, scale)
