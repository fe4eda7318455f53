"""Pins of the parity checker and of the oracle parts that only shape inputs.

CPU only.  The first half shows that the rules every GPU parity test rests on
reject results that are wrong in one place at a time and accept the controls
right next to them: the near-tie window of Eq. encode's argmin, the payload
byte layout, the binary16 norm header, the reconstruction tolerance and the
attention tolerance.  The second half pins, on hand-worked cases, three
oracle functions that were otherwise checked only statistically: the
Roberts-Kronecker direction map of Sec. 3.3 (k >= 4), the empty-cell repair of
the Lloyd-Max polish (App. A codebook-construction table) and the spherical
k-means of App. F Stage 2.
"""
import math
import statistics

import numpy as np
import pytest
import torch

from oracle import codebook as ocb
from oracle import codec as occ
from oracle import philox
from oracle import sublinear as osl
from tests import gpu_helpers as gh


# ----------------------------------------------------------- tie window ----
def test_tie_window_bounds_by_hand():
    """D_min (1 + 1e-6) is the accepted band, on the oracle's float64 D."""
    D = np.array([[[2.0, 2.0 * (1 + 0.9e-6), 2.0 * (1 + 1.1e-6), 2.5]]])
    ref = np.array([[0]])
    ok = [bool(occ.tie_ok(D, ref, np.array([[j]]))[0, 0]) for j in range(4)]
    assert ok == [True, True, False, False]
    # the window is relative: a gap of 1e-7 absolute is outside at D_min = 0.05
    D2 = np.array([[[0.05, 0.05 + 1e-7]]])
    assert not occ.tie_ok(D2, np.array([[0]]), np.array([[1]]))[0, 0]
    # ...and inside at D_min = 0.5
    D3 = np.array([[[0.5, 0.5 + 1e-7]]])
    assert occ.tie_ok(D3, np.array([[0]]), np.array([[1]]))[0, 0]


def test_check_indices_counts_and_rejects():
    D = np.array([[[1.0, 1.0 + 1e-7, 3.0], [4.0, 2.0, 2.0 + 5e-6]]])  # one vector, two blocks
    ref = np.array([[0, 1]])
    assert gh.check_indices(ref, [D], np.array([[0, 1]]), chunk=1) == (2, 0)
    assert gh.check_indices(ref, [D], np.array([[1, 1]]), chunk=1) == (1, 1)  # inside: a tie
    with pytest.raises(AssertionError, match="outside the tie window"):
        gh.check_indices(ref, [D], np.array([[0, 2]]), chunk=1)               # 2.5e-6 outside
    with pytest.raises(AssertionError):
        gh.check_indices(ref, [D], np.array([[2, 1]]), chunk=1)


def _small_problem(N=16, d=16, k=4, n=40, seed=3):
    rng = np.random.default_rng(seed)
    R = ocb.haar_rotation(d, 2).astype(np.float32)
    C = (0.3 * rng.standard_normal((N, k))).astype(np.float32)
    x = rng.standard_normal((n, d)).astype(np.float32).astype(np.float64)
    return x, R, C


def _device_stand_in(x, R, C, N):
    """The result a correct device would return, built by the oracle."""
    idx, h = occ.encode(x, R.astype(np.float64), C.astype(np.float64))
    pay = torch.from_numpy(occ.pack(idx, N))
    nrm = torch.from_numpy(occ.fp16_bits(h).view(np.int16).copy())
    return idx, pay, nrm


def test_check_encode_accepts_the_oracle_result():
    x, R, C = _small_problem()
    _, pay, nrm = _device_stand_in(x, R, C, 16)
    n_exact, n_ties, _, _ = gh.check_encode(x, R, C, 16, pay, nrm)
    assert n_exact == x.shape[0] * 4 and n_ties == 0


def test_check_encode_rejects_a_wrong_index():
    x, R, C = _small_problem()
    idx, _, nrm = _device_stand_in(x, R, C, 16)
    _, _, D = occ.encode(x, R.astype(np.float64), C.astype(np.float64), return_distances=True)
    bad = idx.copy()
    v, m = 7, 2
    bad[v, m] = int(np.argsort(D[v, m])[1])  # the runner-up: a clear gap, not a tie
    assert D[v, m, bad[v, m]] > D[v, m].min() * (1 + 1e-6)
    with pytest.raises(AssertionError, match="outside the tie window"):
        gh.check_encode(x, R, C, 16, torch.from_numpy(occ.pack(bad, 16)), nrm)


def test_check_encode_accepts_an_exact_tie_and_rejects_just_outside():
    """A duplicated codeword makes two indices equally near; moving the copy by
    a hair puts it just outside the window."""
    x, R, C = _small_problem()
    C = C.copy()
    C[11] = C[5]
    idx, _, nrm = _device_stand_in(x, R, C, 16)
    sel = idx == 5
    assert sel.any()
    alt = idx.copy()
    alt[sel] = 11  # the duplicate: D equal to the float64 minimum
    n_exact, n_ties, _, _ = gh.check_encode(x, R, C, 16, torch.from_numpy(occ.pack(alt, 16)), nrm)
    assert n_ties == int(sel.sum()) and n_exact == idx.size - n_ties
    # the same choice against a codebook whose copy sits just outside the window
    _, _, D = occ.encode(x, R.astype(np.float64), C.astype(np.float64), return_distances=True)
    v, m = map(int, np.argwhere(sel)[0])
    C2 = C.copy()
    y = occ.rotate_normalise(x[v:v + 1], R.astype(np.float64), np.linalg.norm(x[v:v + 1], axis=1))
    blk = y[0, 4 * m:4 * m + 4]
    diff = C2[5].astype(np.float64) - blk
    # push codeword 11 outward from the block along c_5 - y by 4e-6 relative in D
    C2[11] = (blk + diff * math.sqrt(1 + 4e-6)).astype(np.float32)
    _, _, D2 = occ.encode(x, R.astype(np.float64), C2.astype(np.float64), return_distances=True)
    assert D2[v, m, 11] > D2[v, m, 5] * (1 + 1e-6)
    one = idx.copy()
    one[v, m] = 11
    with pytest.raises(AssertionError, match="outside the tie window"):
        gh.check_encode(x, R, C2, 16, torch.from_numpy(occ.pack(one, 16)), nrm)


def test_check_encode_rejects_one_flipped_norm_bit():
    x, R, C = _small_problem()
    _, pay, nrm = _device_stand_in(x, R, C, 16)
    for bit in (0, 10, 14):
        bad = nrm.clone()
        bad[3] ^= 1 << bit
        with pytest.raises(AssertionError):
            gh.check_encode(x, R, C, 16, pay, bad)


def test_check_encode_rejects_a_set_padding_bit():
    """N = 8 at d = 16, k = 4: 12 index bits in 2 bytes; the top nibble of byte 1
    must be zero (little-endian bit stream, trailing bits zero)."""
    x, R, C = _small_problem(N=8)
    _, pay, nrm = _device_stand_in(x, R, C, 8)
    gh.check_encode(x, R, C, 8, pay, nrm)
    bad = pay.clone()
    bad[0, 1] |= 0x80
    with pytest.raises(AssertionError):
        gh.check_encode(x, R, C, 8, bad, nrm)


def test_check_recon_tolerance_scales_with_the_norm():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((5, 8))
    hdr = np.array([0.5, 1.0, 3.0, 100.0, 1e3])
    gh.check_recon(ref.astype(np.float64).copy(), ref, hdr)
    for v, scale in ((0, 1.0), (3, 100.0), (4, 1e3)):
        ok = ref.copy()
        ok[v, 2] += 0.5 * 1e-5 * scale
        gh.check_recon(ok, ref, hdr)
        bad = ref.copy()
        bad[v, 2] += 2.0 * 1e-5 * scale
        with pytest.raises(AssertionError, match="max err/tol"):
            gh.check_recon(bad, ref, hdr)


def test_check_attention_rejects_a_head_off_by_3e_3():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((3, 8, 64))
    assert gh.check_attention(ref.copy(), ref) == 0.0
    close = ref.copy()
    close[1, 5] *= 1 + 1e-3
    assert gh.check_attention(close, ref) <= 1.01e-3
    bad = ref.copy()
    bad[1, 5] *= 1 + 3e-3
    with pytest.raises(AssertionError, match="max rel l2"):
        gh.check_attention(bad, ref)
    # the elementwise bound catches one element off by 3e-3 of the head's max
    spike = ref.copy()
    spike[2, 0, 7] += 3e-3 * np.abs(ref[2, 0]).max()
    with pytest.raises(AssertionError):
        gh.check_attention(spike, ref)


# --------------------------------------------- Roberts-Kronecker (k >= 4) ---
def test_roberts_kronecker_k4_by_hand():
    """Sec. 3.3: xi_{n,j} = {(n - 1/2) phi_4^-j}, phi_4^5 = phi_4 + 1, then the
    standard-normal quantile, then the projection to S^3."""
    phi = ocb.roberts_phi(4)
    assert abs(phi - 1.1673039782614187) < 1e-13   # the root of x^5 = x + 1
    xi = ocb.kronecker_points(4, 6)
    # n = 1: half the generator (an off-by-1/2 in n, or j counted from 0, fails)
    step = np.array([phi ** -1, phi ** -2, phi ** -3, phi ** -4])
    assert np.allclose(xi[0], 0.5 * step, atol=1e-15, rtol=0)
    assert np.allclose(xi[0], [0.42833744, 0.36694593, 0.31435336, 0.26929863], atol=1e-8)
    # additive recurrence: xi_{n+1} = {xi_n + phi^-j}
    for n in range(5):
        assert np.allclose(np.mod(xi[n] + step, 1.0), xi[n + 1], atol=1e-12, rtol=0)
    # directions: Phi^-1 of the points (standard library quantile), normalised
    u = ocb.directions(4, 6)
    nd = statistics.NormalDist()
    for n in range(6):
        g = np.array([nd.inv_cdf(float(t)) for t in xi[n]])
        assert np.allclose(u[n], g / np.linalg.norm(g), atol=1e-12, rtol=0)
    # the first direction by hand: Phi^-1(0.4283..), .. all negative (< 1/2)
    assert np.all(u[0] < 0)
    # continuing the sequence (App. E fresh sets) is an index offset
    assert np.allclose(ocb.kronecker_points(4, 3, offset=3), xi[3:6], atol=1e-12, rtol=0)


# ------------------------------------------------------- empty-cell repair ---
def test_lloyd_round_repairs_empty_cells_by_hand():
    """Two occupied cells and two empty ones.  Cell 0 has 2 samples and the
    larger within-cell error (0.08), cell 1 has 3 samples and 0.02: the first
    empty cell takes half of cell 0 (the largest error, not the most members),
    leaving it one member, so the second empty cell must take cell 1."""
    x = np.array([[1.0, 0.0], [1.0, 0.4], [-1.0, 0.0], [-1.0, -0.1], [-1.0, 0.1]])
    c = np.array([[1.0, 0.1], [-1.0, 0.05], [5.0, 5.0], [6.0, -6.0]])
    seed = 9
    out, events = ocb.lloyd_round(x, c, seed, repair_events=0)
    assert events == 2

    def unit(i):
        g = philox.normals(seed, philox.TAG_REPAIR, 2 * i, 2)
        return g / np.linalg.norm(g)

    mean0, mean1 = np.array([1.0, 0.2]), np.array([-1.0, 0.0])
    d0 = 1e-2 * math.sqrt(0.08 / 2) * unit(0)     # rms error of cell 0: 0.2
    d1 = 1e-2 * math.sqrt(0.02 / 3) * unit(1)     # cell 1's error is untouched
    assert np.allclose(out[2], mean0 + d0, atol=1e-15, rtol=0)
    assert np.allclose(out[0], mean0 - d0, atol=1e-15, rtol=0)
    assert np.allclose(out[3], mean1 + d1, atol=1e-15, rtol=0)
    assert np.allclose(out[1], mean1 - d1, atol=1e-15, rtol=0)
    # the input codebook is not modified
    assert c[2, 0] == 5.0


def test_lloyd_round_plain_centroid_step():
    """No empty cell: each codeword moves to the mean of its cell (Lloyd's
    centroid condition) and no repair draw is spent."""
    x = np.array([[0.0, 0.0], [0.2, 0.0], [1.0, 1.0], [1.0, 1.4]])
    c = np.array([[0.1, 0.1], [0.9, 1.1]])
    out, events = ocb.lloyd_round(x, c, 1, repair_events=5)
    assert events == 5
    assert np.allclose(out, [[0.1, 0.0], [1.0, 1.2]], atol=1e-15, rtol=0)


# ------------------------------------------ spherical k-means (App. F Stage 2) ---
def test_parent_groups_on_a_symmetric_set():
    """Eight planar directions in four tight pairs (0/10, 90/100, 180/190,
    270/280 degrees): started from every second direction, the parents are
    the pairs and their mean directions the bisectors (5, 95, 185, 275)."""
    ang = np.deg2rad([0, 10, 90, 100, 180, 190, 270, 280])
    U = np.stack([np.cos(ang), np.sin(ang)], axis=1)
    g, mu = osl.parent_groups(U, 4, rounds=3)
    assert g.tolist() == [0, 0, 1, 1, 2, 2, 3, 3]
    want = np.deg2rad([5, 95, 185, 275])
    assert np.allclose(mu, np.stack([np.cos(want), np.sin(want)], axis=1), atol=1e-12, rtol=0)
    assert np.allclose(np.linalg.norm(mu, axis=1), 1.0)


def test_parent_groups_assign_by_largest_inner_product():
    """Three directions near +x and one near -x with K = 2 started from
    codewords 0 and 2: the -x direction must leave parent 1's +x start."""
    ang = np.deg2rad([0, 20, 40, 180])
    U = np.stack([np.cos(ang), np.sin(ang)], axis=1)
    g, mu = osl.parent_groups(U, 2, rounds=4)
    # iteration 1 (starts at 0 and 40 degrees): {0, 20} and {40, 180} (20 is
    # equidistant and goes to the first parent); iteration 2: the second mean points
    # to 110 degrees, so 40 moves over and the parents settle at {0, 20, 40}
    # (mean 20 degrees) and {180}.  Assigning by the smallest inner product
    # would pair 180 with the +x directions instead.
    assert g[3] != g[0] and g[0] == g[1] == g[2]
    assert np.allclose(mu[g[3]], [-1.0, 0.0], atol=1e-12)
    assert np.allclose(mu[g[0]], [math.cos(math.radians(20)), math.sin(math.radians(20))],
                       atol=1e-12)
