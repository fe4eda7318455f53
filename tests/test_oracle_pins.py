"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test names the passage it follows.  None of them re-derives an expected
value with the oracle's own routine: expected values are printed numbers of
the paper (tests/golden/), closed forms, hand-worked cases, brute force on
tiny inputs, or an independent formula for the same quantity.
"""
import math
import os

import numpy as np
import pytest
from scipy.special import betaincinv, gammaln

from oracle import attention as oat
from oracle import codebook as ocb
from oracle import codec as occ
from oracle import fileio as ofio
from oracle import philox
from oracle import sublinear as osl

from _fixtures import oracle_codebook, oracle_rotation, read_table

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------ generator ---
def test_philox_known_answers():
    """Philox4x32-10 reproduces the published Random123 known-answer vectors."""
    for row in read_table(os.path.join(GOLDEN, "philox4x32_10_kat.txt")):
        v = [int(x, 16) for x in row]
        out = philox.philox4x32_10(tuple(v[0:4]), tuple(v[4:6]))
        assert [int(o) for o in out] == v[6:10]


def test_normal_stream_moments():
    z = philox.normals(123, 7, 0, 400000)
    assert abs(z.mean()) < 5 / math.sqrt(4e5)
    assert abs(z.var() - 1.0) < 5 * math.sqrt(2 / 4e5)
    assert abs((z ** 4).mean() - 3.0) < 0.05
    # a window of the stream equals the same normals drawn from a later start
    assert np.array_equal(philox.normals(123, 7, 1001, 10), z[1001:1011])


# ------------------------------------------------------------- rotation ---
def test_rotation_orthogonal_after_fp32_rounding():
    """P1: the stored fp32 Pi is orthogonal to 1e-6 (evaluated in fp64)."""
    for d in (64, 128):
        R = oracle_rotation(d).astype(np.float64)
        assert np.abs(R.T @ R - np.eye(d)).max() <= 1e-6
        assert np.abs(R @ R.T - np.eye(d)).max() <= 1e-6


def test_rotation_is_qr_with_positive_diagonal():
    """Haar construction (Mezzadri): Q^T G is upper triangular with diag > 0."""
    d = 16
    g = philox.normals(5, philox.TAG_ROTATION, 0, d * d).reshape(d, d)
    Q = ocb.haar_from_normals(g)
    Rm = Q.T @ g
    assert np.abs(np.tril(Rm, -1)).max() < 1e-12
    assert (np.diag(Rm) > 0).all()


def test_rotation_entries_have_haar_moments():
    """A Haar orthogonal d x d matrix has E Pi_ij = 0 and E Pi_ij^2 = 1/d."""
    d, reps = 6, 3000
    acc1 = np.zeros((d, d))
    acc2 = np.zeros((d, d))
    for s in range(reps):
        g = philox.normals(s, philox.TAG_ROTATION, 0, d * d).reshape(d, d)
        Q = ocb.haar_from_normals(g)
        acc1 += Q
        acc2 += Q * Q
    assert np.abs(acc1 / reps).max() < 5 * math.sqrt(1 / d / reps)
    assert np.abs(acc2 / reps - 1.0 / d).max() < 0.02


# --------------------------------------------------------------- source ---
@pytest.mark.parametrize("d,k", [(64, 4), (64, 2), (128, 4), (64, 8)])
def test_spherical_beta_radial_moments(d, k):
    """P2, Lemma 1 / Eq. radial_law: R^2 ~ Beta(k/2, (d-k)/2), E R^2 = k/d,
    Var R^2 = 2k(d-k) / (d^2 (d+2))."""
    n = 200000
    x = ocb.sample_source(d, k, n, seed=11)
    r2 = (x * x).sum(axis=1)
    var = 2 * k * (d - k) / (d * d * (d + 2))
    assert abs(r2.mean() - k / d) < 5 * math.sqrt(var / n)
    assert abs(r2.var() - var) < 0.03 * var
    # X / R uniform on the sphere: E[X X^T] = (1/d) I (isotropic block)
    cov = x.T @ x / n
    assert np.abs(cov - np.eye(k) / d).max() < 6 * math.sqrt(2.0 / n) / d


def test_scalar_marginal_k1():
    """App. B: the k = 1 marginal has E X = 0 and Var X = 1/d."""
    d, n = 64, 200000
    x = ocb.sample_source(d, 1, n, seed=3)[:, 0]
    assert abs(x.mean()) < 5 * math.sqrt(1 / d / n)
    assert abs(x.var() - 1 / d) < 0.02 / d


# ---------------------------------------------------------------- radii ---
@pytest.mark.parametrize("d", [16, 64, 128])
def test_k2_radii_closed_form_equals_beta_quantiles(d):
    """P3: Eq. radii_k2 is Eq. radii_main at k = 2 (beta_{d,2} = d/4)."""
    N = 16
    q = (np.arange(1, N + 1) - 0.5) / N
    via_beta = np.sqrt(betaincinv(1.0, d / 4.0, q))
    assert ocb.beta_dk(d, 2) == pytest.approx(d / 4.0)
    assert np.allclose(ocb.radii(d, 2, N), via_beta, rtol=0, atol=1e-14)


def test_radii_follow_companded_beta_law():
    """Eq. radii_main: r_n^2 are the midpoint quantiles of Beta(k/2, beta_dk):
    checked through the regularised incomplete beta function itself."""
    from scipy.special import betainc
    d, k, N = 64, 4, 32
    r = ocb.radii(d, k, N)
    assert np.all(np.diff(r) > 0) and r[0] > 0 and r[-1] < 1
    q = betainc(k / 2.0, ocb.beta_dk(d, k), r ** 2)
    assert np.allclose(q, (np.arange(1, N + 1) - 0.5) / N, atol=1e-12)


# ----------------------------------------------------------- directions ---
def test_directions_unit_and_golden_angle():
    """Sec. 3.3: unit directions; k = 2 spiral steps by 2 pi (1 - 1/phi)."""
    for k in (2, 3, 4, 8):
        u = ocb.directions(k, 64)
        assert np.allclose(np.linalg.norm(u, axis=1), 1.0, atol=1e-14)
    u = ocb.directions(2, 8)
    ang = np.arctan2(u[:, 1], u[:, 0])
    step = np.mod(np.diff(ang), 2 * np.pi)
    assert np.allclose(step, np.mod(2 * np.pi * (1 - 2 / (1 + math.sqrt(5))), 2 * np.pi))
    # k = 3: equal-area latitude bands z_n = 1 - (2n - 1)/M (App. E)
    u3 = ocb.directions(3, 10)
    assert np.allclose(u3[:, 2], 1 - (2 * np.arange(1, 11) - 1) / 10)


def test_roberts_phi_root():
    """phi_k is the positive root of phi^(k+1) = phi + 1; phi_1 is the golden ratio."""
    assert ocb.roberts_phi(1) == pytest.approx((1 + math.sqrt(5)) / 2, abs=1e-12)
    for k in (4, 8, 16):
        p = ocb.roberts_phi(k)
        assert abs(p ** (k + 1) - p - 1) < 1e-12


# ---------------------------------------------------------------- Lloyd ---
def test_scalar_two_level_closed_form():
    """P4: k = 1, N = 2 optimum is +/- E|X| with E|X| = Gamma(d/2) / (sqrt(pi)
    Gamma((d+1)/2)); normalised distortion d (1/d - E|X|^2) = 0.358387 at d=64."""
    d = 64
    C, _ = oracle_codebook(d, 1, 2, M=100000)
    ex = math.exp(gammaln(d / 2) - gammaln((d + 1) / 2)) / math.sqrt(math.pi)
    assert ex == pytest.approx(0.100126, abs=1e-6)
    lv = np.sort(C[:, 0])
    assert lv[0] == pytest.approx(-ex, abs=1.5e-3) and lv[1] == pytest.approx(ex, abs=1.5e-3)
    mse = ocb.mse_on(C, d, 1, 200000, seed=9)
    assert d * mse == pytest.approx(d * (1 / d - ex * ex), rel=0.01)
    assert d * (1 / d - ex * ex) == pytest.approx(0.358387, abs=1e-6)


@pytest.mark.parametrize("N", [4, 8, 16])
def test_scalar_lloyd_matches_turboquant_table(N):
    """P5: k = 1 (scalar TurboQuant, Sec. 3.2 remark) reproduces the printed
    TurboQuant NMSE of App. G at b = 2, 3, 4 within 0.15 dB."""
    d = 64
    want = {int(r[2]): float(r[4]) for r in read_table(os.path.join(GOLDEN, "paper_table2_nmse.txt"))
            if r[0] == "turboquant"}[N]
    C, _ = oracle_codebook(d, 1, N, M=100000)
    got = ocb.nmse_db(ocb.mse_on(C, d, 1, 200000, seed=9), d, 1)
    assert abs(got - want) < 0.15, (got, want)


def test_dominance_k2_over_scalar():
    """P7, Thm. 2: at b = 2, the k = 2 code (N = 16) beats the scalar (N = 4)."""
    d = 64
    C2, _ = oracle_codebook(d, 2, 16, M=100000)
    C1, _ = oracle_codebook(d, 1, 4, M=100000)
    per_coord_2 = ocb.mse_on(C2, d, 2, 200000, seed=9) / 2
    per_coord_1 = ocb.mse_on(C1, d, 1, 200000, seed=9)
    assert per_coord_2 < per_coord_1


def test_distortion_non_increasing_in_N():
    """P8: held-out MSE is non-increasing along N = 2, 4, ..., 64 (k = 2)."""
    d, k = 64, 2
    m = [ocb.mse_on(oracle_codebook(d, k, N, M=30000, restarts=2)[0], d, k, 100000, seed=9)
         for N in (2, 4, 8, 16, 32, 64)]
    assert all(b <= a for a, b in zip(m, m[1:])), m


def test_lloyd_trace_restarts_and_empty_cells():
    """App. A table: each restart's D(C) is a training MSE; the kept one is the
    minimum.  Heavily over-provisioned N forces empty-cell repairs."""
    C, D, trace = ocb.lloyd_max(64, 2, 64, seed=3, M=300, restarts=3, iters=6,
                                return_trace=True)
    assert D == min(trace)
    x = ocb.sample_source(64, 2, 300, 3, philox.TAG_TRAIN)
    dist = ((x[:, None, :] - C[None]) ** 2).sum(-1).min(1).mean()
    assert dist == pytest.approx(D, rel=1e-12)


# ------------------------------------------------ starting-codebook variants ---
@pytest.mark.parametrize("k", [1, 2, 4, 8])
def test_multishell_reduces_to_the_single_family_designs(k):
    """App. E Eq. multishell: with M_a = 1 every shell holds one direction and
    C(N, 1) is the N-radius codebook of Eq. radii_main; with S = 1 it is the
    whole direction set on the median Beta radius (q = 1/2)."""
    d, N = 64, 32
    assert np.array_equal(ocb.multishell_codebook(d, k, N, 1), ocb.initial_codebook(d, k, N))
    beta = k / (k + 2) * (d - k - 2) / 2 + 1
    r_med = math.sqrt(betaincinv(k / 2, beta, 0.5))
    one = ocb.multishell_codebook(d, k, 1, N)
    assert np.allclose(np.linalg.norm(one, axis=1), r_med, rtol=1e-12, atol=0)
    assert np.allclose(one / r_med, ocb.directions(k, N), rtol=0, atol=1e-12)


def test_multishell_k3_bands_and_golden_azimuth():
    """App. E Eq. fib_sphere_3d per shell: the latitudes of each shell are M_a
    equal-area bands (equally spaced z, symmetric about 0), the radii are the
    Beta quantiles at q_s = (s - 1/2)/S, and the azimuth advances by the golden
    angle 2 pi (1 - 1/phi) from every codeword to the next, across shells too."""
    d, k, S, Ma = 64, 3, 4, 32
    c = ocb.multishell_codebook(d, k, S, Ma)
    beta = k / (k + 2) * (d - k - 2) / 2 + 1
    golden = 2 * math.pi * (1 - 2 / (1 + math.sqrt(5)))
    for s in range(S):
        blk = c[s * Ma:(s + 1) * Ma]
        r = math.sqrt(betaincinv(k / 2, beta, (s + 0.5) / S))
        assert np.allclose(np.linalg.norm(blk, axis=1), r, rtol=1e-12, atol=0)
        z = np.sort(blk[:, 2] / r)
        assert np.allclose(np.diff(z), 2 / Ma, atol=1e-12) and abs(z.sum()) < 1e-12
    az = np.arctan2(c[:, 1], c[:, 0])
    step = np.mod(np.diff(az) - golden + math.pi, 2 * math.pi) - math.pi
    assert np.abs(step).max() < 1e-9


def test_multishell_search_lowers_k3_training_mse():
    """App. E: at k = 3 and moderate d the factor-pair search picks a few
    shells (S of order d^(1/3), not the N shells of Eq. radii_main) and lowers
    the training MSE, before and after the polish, by up to about 0.3 dB."""
    d, k, N, M = 64, 3, 128, 30 * 128
    x = ocb.sample_source(d, k, M, 1, philox.TAG_TRAIN)
    S, c = ocb.choose_multishell(d, k, N, x)
    assert 2 <= S <= 16
    e_beta = ((x[:, None, :] - ocb.initial_codebook(d, k, N)[None]) ** 2).sum(-1).min(1).mean()
    e_multi = ((x[:, None, :] - c[None]) ** 2).sum(-1).min(1).mean()
    assert e_multi < e_beta
    _, m_beta = ocb.lloyd_max(d, k, N, 1, M, 2, 20)
    _, m_multi, shells = ocb.lloyd_max(d, k, N, 1, M, 2, 20, init="multishell",
                                       return_shells=True)
    assert shells == S
    gain_db = 10 * math.log10(m_beta / m_multi)
    assert 0 < gain_db < 0.5, gain_db


def test_single_shell_shortcut_reaches_the_beta_optimum():
    """App. D: the source concentrates at radius sqrt(k/d) (E R^2 = k/d
    exactly), and the polished single-shell codebook reaches the distortion of
    the polished Beta-quantile codebook (difference O(1/d))."""
    d, k, N = 256, 4, 64
    c = ocb.single_shell_codebook(d, k, N)
    assert np.allclose(np.linalg.norm(c, axis=1), math.sqrt(k / d), rtol=1e-12, atol=0)
    got = []
    for init in ("beta", "shell"):
        C, _ = ocb.lloyd_max(d, k, N, 1, 20000, 1, 20, init=init)
        got.append(ocb.mse_on(C, d, k, 100000, seed=9))
    assert abs(got[1] - got[0]) / got[0] < 0.01, got


@pytest.mark.parametrize("d", [16, 32])
def test_full_vector_code_two_codewords_closed_form(d):
    """Sec. 5 (full-vector code, k = d): the source is the whole unit vector, so
    every antipodal pair +/- a u has distortion 1 - 2 a E|y_1| + a^2 whatever
    the direction u; the optimum a = E|y_1| = Gamma(d/2) / (sqrt(pi)
    Gamma((d+1)/2)) gives 1 - E|y_1|^2.  Lloyd at N = 2 must land there."""
    ex = math.exp(gammaln(d / 2) - gammaln((d + 1) / 2)) / math.sqrt(math.pi)
    C, _ = ocb.lloyd_max(d, d, 2, 1, 40000, 1, 15)
    n = np.linalg.norm(C, axis=1)
    assert np.allclose(n, ex, rtol=0.05), (n, ex)
    assert np.linalg.norm(C.sum(0)) < 0.1 * ex  # antipodal
    held = ocb.mse_on(C, d, d, 100000, seed=9)
    # held-out noise: per-sample sd 2 E|y_1| sd|y_1| <= 0.06, over 1e5 samples
    assert abs(held - (1 - ex * ex)) < 1e-3, (held, 1 - ex * ex)


# ---------------------------------------------------------------- codec ---
def _codec_nmse(d, k, N, C, n=20000, law="normal"):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((n, d))
    if law == "lognormal_outlier":
        sig = np.exp(0.5 * rng.standard_normal(d))
        sig[rng.permutation(d)[:2]] *= 10
        x = x * sig
    R = oracle_rotation(d)
    idx, h = occ.encode(x, R, C)
    xh = occ.decode(idx, h, R, C)
    return 10 * math.log10(((x - xh) ** 2).sum() / (x * x).sum())


@pytest.mark.parametrize("k,N,M,restarts", [(2, 64, 100000, 2), (4, 256, 40000, 1)])
def test_codec_reproduces_table2_nmse(k, N, M, restarts):
    """P6: the whole oracle codec (norm, rotation, argmin, decoder) on synthetic
    caches reproduces the printed FibQuant NMSE of App. G within 0.35 dB."""
    d = 64
    want = {(int(r[1]), int(r[2])): float(r[4])
            for r in read_table(os.path.join(GOLDEN, "paper_table2_nmse.txt"))
            if r[0] == "fibquant"}[(k, N)]
    C, _ = oracle_codebook(d, k, N, M=M, restarts=restarts)
    got = _codec_nmse(d, k, N, C)
    assert abs(got - want) < 0.35, (got, want)


def test_universality_heavy_tailed_channels():
    """Thm. 1: norm + Haar rotation make the distortion independent of the
    input law (outlier channels vs isotropic Gaussian)."""
    d, k, N = 64, 2, 16
    C, _ = oracle_codebook(d, k, N, M=100000)
    a = _codec_nmse(d, k, N, C, n=20000)
    b = _codec_nmse(d, k, N, C, n=20000, law="lognormal_outlier")
    assert abs(a - b) < 0.1, (a, b)


def test_encode_orientation_and_normalisation_by_hand():
    """Sec. 3.1: y = Pi x / ||x|| with y_i = sum_j Pi_ij x_j (row-major Pi).
    A cyclic-shift Pi and a hand-picked codebook fix the expected indices."""
    d, k = 4, 2
    Pi = np.zeros((d, d))
    for i in range(d):
        Pi[i, (i + 1) % d] = 1.0  # (Pi x)_i = x_{i+1}
    C = np.array([[0.0, 0.0], [0.8, 0.0], [0.0, 0.8], [-0.8, 0.0]])
    x = np.array([0.0, 3.0, 0.0, 0.0])  # ||x|| = 3, y = (1, 0, 0, 0)
    idx, h = occ.encode(x[None], Pi, C)
    assert idx.tolist() == [[1, 0]]
    assert float(h[0]) == 3.0
    x = np.array([0.0, 0.0, 0.0, 2.0])  # y = (0, 0, 1, 0)
    idx, _ = occ.encode(x[None], Pi, C)
    assert idx.tolist() == [[0, 1]]
    # the transpose orientation would give y = (0, 0, 0, 1) -> [[0, 2]]
    y = occ.rotate_normalise(np.array([[1.0, 2.0, 2.0, 4.0]]), Pi, np.array([5.0]))
    assert np.allclose(y, [[0.4, 0.4, 0.8, 0.2]])


def test_normalisation_uses_exact_norm():
    """Reading Q1: the unit vector is formed with the unrounded norm."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((50, 64)) * 37.3
    nu, h = occ.norms(x)
    y = occ.rotate_normalise(x, oracle_rotation(64), nu)
    assert np.allclose(np.linalg.norm(y, axis=1), 1.0, atol=1e-14)
    assert np.abs(h.astype(np.float64) / nu - 1).max() > 1e-6  # header really is rounded


def test_norm_header_round_to_nearest_even_by_hand():
    """fp16 header (Sec. 3.1) rounded to nearest, ties to even (hand-worked bits)."""
    cases = [
        (1.0 + 2 ** -11, 0x3C00),            # midpoint 1 | 1+2^-10 -> even (1.0)
        (1.0 + 3 * 2 ** -11, 0x3C02),        # midpoint -> even mantissa 2
        (1.0 + 2 ** -11 + 2 ** -30, 0x3C01),  # just above the midpoint
        (65504.0, 0x7BFF), (65519.0, 0x7BFF), (65520.0, 0x7C00),  # overflow to inf
        (2.0 ** -24, 0x0001), (2.0 ** -25, 0x0000), (3 * 2.0 ** -25, 0x0002),  # subnormals
    ]
    for val, bits in cases:
        _, h = occ.norms(np.array([[val, 0.0, 0.0, 0.0]]))
        assert int(occ.fp16_bits(h)[0]) == bits, (val, hex(int(occ.fp16_bits(h)[0])))


def test_zero_vector_and_lowest_index_ties():
    """Reading Q2 (zero vector -> header 0, indices 0, decodes to 0) and Q4
    (exact ties go to the lowest index)."""
    C = np.array([[0.5, 0.0], [0.5, 0.0], [0.0, 0.5], [0.0, 0.5]])
    Pi = np.eye(4)
    idx, h = occ.encode(np.array([[0.0, 0, 0, 0], [1.0, 0, 0, 1]]), Pi, C)
    assert idx.tolist() == [[0, 0], [0, 2]]
    assert float(h[0]) == 0.0
    assert np.all(occ.decode(idx[:1], h[:1], Pi, C) == 0)


def test_exhaustive_product_search_tiny():
    """P9: the per-block argmin equals the brute-force minimum over all N^(d/k)
    concatenated codewords of ||y - y_hat||^2 (computed on the whole vector)."""
    import itertools
    rng = np.random.default_rng(2)
    for d, k, N in [(4, 2, 4), (6, 2, 8), (8, 4, 8), (6, 3, 4)]:
        C = rng.standard_normal((N, k)) * 0.4
        Pi = oracle_rotation(d) if d in (64, 128) else ocb.haar_rotation(d, 9)
        x = rng.standard_normal((30, d))
        idx, h = occ.encode(x, Pi, C)
        nu = np.linalg.norm(x, axis=1)
        y = (x / nu[:, None]) @ Pi.T
        for v in range(x.shape[0]):
            best, arg = np.inf, None
            for combo in itertools.product(range(N), repeat=d // k):
                e = np.linalg.norm(y[v] - np.concatenate([C[c] for c in combo])) ** 2
                if e < best:
                    best, arg = e, combo
            assert tuple(idx[v]) == arg


def test_scalar_k1_equals_per_coordinate_quantiser():
    """k = 1 reduces to the scalar product quantiser: each rotated coordinate is
    mapped to its nearest level, found here by sorting levels and comparing
    against decision thresholds at the midpoints."""
    d = 64
    C, _ = oracle_codebook(d, 1, 8, M=100000)
    rng = np.random.default_rng(4)
    x = rng.standard_normal((200, d))
    idx, _ = occ.encode(x, oracle_rotation(d), C)
    nu = np.linalg.norm(x, axis=1)
    y = (x / nu[:, None]) @ oracle_rotation(d).astype(np.float64).T
    order = np.argsort(C[:, 0])
    levels = C[order, 0]
    thr = 0.5 * (levels[1:] + levels[:-1])
    want = order[np.searchsorted(thr, y)]
    assert np.array_equal(idx, want)


def test_decoded_blocks_lie_in_their_voronoi_cells():
    """BJ invariant: decode(encode(x)) lies in the cell of each chosen codeword:
    checked in the expanded form ||c||^2 - 2<y, c> (a different formula from the
    encoder's direct distances), to a 1e-12 window."""
    d, k, N = 64, 4, 256
    C = oracle_codebook(d, 4, 256, M=40000, restarts=1)[0]
    R = ocb.haar_rotation(d, 2)  # float64, orthogonal to rounding
    rng = np.random.default_rng(8)
    x = rng.standard_normal((300, d)) * 3
    idx, h = occ.encode(x, R, C)
    xh = occ.decode(idx, h, R, C)
    yhat = (xh / h.astype(np.float64)[:, None]) @ R.T  # rotate back, strip the header
    assert np.allclose(yhat.reshape(300, d // k, k), C[idx], atol=1e-12)
    y = (x / np.linalg.norm(x, axis=1)[:, None]) @ R.T
    yb = y.reshape(300, d // k, k)
    score = (C * C).sum(1)[None, None, :] - 2 * np.einsum("vmi,ni->vmn", yb, C)
    chosen = np.take_along_axis(score, idx[..., None], axis=-1)[..., 0]
    assert np.all(chosen <= score.min(axis=-1) + 1e-12)


def test_random_access_row_decode():
    """P11: decoding one token alone equals that row of the full decode."""
    d = 64
    C = oracle_codebook(d, 2, 16, M=20000, restarts=1)[0]
    R = oracle_rotation(d)
    x = np.random.default_rng(3).standard_normal((40, d))
    idx, h = occ.encode(x, R, C)
    full = occ.decode(idx, h, R, C)
    for t in (0, 17, 39):
        # BLAS may block one row differently from forty: equal to rounding
        assert np.allclose(occ.decode(idx[t:t + 1], h[t:t + 1], R, C)[0], full[t],
                           rtol=0, atol=1e-13)


# ----------------------------------------------------------- bit layout ---
def test_bitpack_hand_worked_examples():
    for row in read_table(os.path.join(GOLDEN, "bitpack_example.txt")):
        w = int(row[0])
        idx = np.array([[int(v) for v in row[1].split(",")]])
        want = [int(v, 16) for v in row[2].split(",")]
        got = occ.pack(idx, 2 ** w)
        assert got[0].tolist() == want
        assert np.array_equal(occ.unpack(got, idx.shape[1], 2 ** w), idx)


def test_payload_size_and_paper_byte_accounting():
    """P12: fixed rate (d log2 N)/k bits (Sec. 3.1); the paper's cache size and
    compression ratios follow from it."""
    rows = read_table(os.path.join(GOLDEN, "paper_compression.txt"))
    for r in rows:
        if r[0] == "gpt2_cache_mb":
            L, H, T, d, want = int(r[1]), int(r[2]), int(r[3]), int(r[4]), float(r[5])
            assert L * H * T * 2 * d * 2 / 1e6 == pytest.approx(want, abs=0.005)
        elif r[0] == "ratio_with_norm":
            d, k, N, want = int(r[1]), int(r[2]), int(r[3]), float(r[4])
            bits = (d // k) * occ.index_bits(N) + 16
            assert 16 * d / bits == pytest.approx(want, abs=0.05)
        elif r[0] == "ratio_no_norm":
            k, N, want = int(r[1]), int(r[2]), float(r[3])
            b = occ.index_bits(N) / k
            assert 16 / b == pytest.approx(want, abs=0.05)
    # the workloads' payloads: 16, 16, 24, 4, 6 and 48 bytes
    for (d, k, N, P) in [(64, 2, 16, 16), (64, 4, 256, 16), (64, 2, 64, 24), (64, 8, 16, 4),
                         (64, 8, 64, 6), (128, 4, 4096, 48)]:
        assert occ.payload_bytes(d, k, N) == P


# ------------------------------------------------------------ attention ---
def test_attention_special_cases():
    """P10, Eq. lattn: T = 1 gives the value; identical keys give the mean
    value; q = 0 gives the mean value; T = 0 gives zero."""
    rng = np.random.default_rng(0)
    d, G, T = 64, 3, 9
    q = rng.standard_normal((G, d))
    V = rng.standard_normal((T, d))
    K = rng.standard_normal((T, d))
    assert np.allclose(oat.attention(q, K[:1], V[:1]), np.repeat(V[:1], G, 0), atol=1e-15)
    Kid = np.repeat(K[:1], T, 0)
    assert np.allclose(oat.attention(q, Kid, V), np.repeat(V.mean(0, keepdims=True), G, 0))
    assert np.allclose(oat.attention(np.zeros((G, d)), K, V),
                       np.repeat(V.mean(0, keepdims=True), G, 0))
    assert np.all(oat.attention(q, K[:0], V[:0]) == 0)


def test_attention_scale_is_inverse_sqrt_d_by_hand():
    """Eq. lattn scale 1/sqrt(d): keys whose dot products with q differ by
    sqrt(d) ln 3 get softmax weights 3/4 and 1/4."""
    d = 64
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    K = np.zeros((2, d))
    K[0, 0] = math.sqrt(d) * math.log(3.0)
    V = np.zeros((2, d))
    V[0, 1] = 1.0
    V[1, 2] = 1.0
    o = oat.attention(q, K, V)
    assert o[0, 1] == pytest.approx(0.75, abs=1e-14) and o[0, 2] == pytest.approx(0.25, abs=1e-14)


def test_attention_stable_and_permutation_invariant():
    rng = np.random.default_rng(1)
    d, T = 64, 50
    q = rng.standard_normal((2, d)) * 300
    K = rng.standard_normal((T, d)) * 300
    V = rng.standard_normal((T, d))
    o = oat.attention(q, K, V)
    assert np.isfinite(o).all()
    perm = rng.permutation(T)
    assert np.allclose(oat.attention(q, K[perm], V[perm]), o, atol=1e-12)


# ----------------------------------------------------------------- file ---
def test_codebook_file_roundtrip_and_corruption():
    C = np.arange(32, dtype=np.float32).reshape(16, 2) / 40
    Pi = np.eye(8, dtype=np.float32)
    blob = ofio.dumps(8, 2, 16, C, Pi, (2, 1))
    got = ofio.loads(blob)
    assert np.array_equal(got["C"], C) and np.array_equal(got["Pi"], Pi)
    assert got["seeds"] == (2, 1) and (got["d"], got["k"], got["N"]) == (8, 2, 16)
    bad = bytearray(blob)
    bad[50] ^= 1
    with pytest.raises(ValueError):
        ofio.loads(bytes(bad))
    # FNV-1a 64 of the empty string and of "a" (published test values)
    assert ofio.fnv1a64(b"") == 0xCBF29CE484222325
    assert ofio.fnv1a64(b"a") == 0xAF63DC4C8601EC8C


# ------------------------------------------- Mahalanobis objective (Sec. 3) ---
@pytest.mark.parametrize("w", [4.0, 0.25])
def test_mahalanobis_two_codewords_closed_form(w):
    """Task-weighted Lloyd (Sec. 3, after Eq. lattn) with M = diag(w, 1) at
    k = 2, N = 2: the source is isotropic in the plane, so the optimum splits
    along the heavier axis, codewords +/- E|y_1| e, and the M-distortion is
    max(w, 1) (1/d - E|y_1|^2) + min(w, 1) / d."""
    d, k = 16, 2
    ex = math.exp(gammaln(d / 2) - gammaln((d + 1) / 2)) / math.sqrt(math.pi)
    C, D = ocb.lloyd_max(d, k, 2, 1, 60000, 1, 15, metric=np.diag([w, 1.0]))
    axis = 0 if w > 1 else 1
    assert np.allclose(np.abs(C[:, axis]), ex, rtol=0.05) and np.abs(C[:, 1 - axis]).max() < 0.02
    want = max(w, 1.0) * (1 / d - ex * ex) + min(w, 1.0) / d
    x = ocb.sample_source(d, k, 200000, 9, philox.TAG_HELDOUT)
    held = ocb.nearest(x, C, np.diag([w, 1.0]))[1].mean()  # held-out M-distortion
    assert held == pytest.approx(want, rel=3e-3)


def test_mahalanobis_identity_and_scaled_metrics():
    """M = I is the plain objective (same codebook, same MSE); M = a I moves
    no assignment, so the codebook is the same and the MSE scales by a."""
    d, k, N = 64, 2, 16
    C, D = ocb.lloyd_max(d, k, N, 1, 20000, 2, 6)
    C1, D1 = ocb.lloyd_max(d, k, N, 1, 20000, 2, 6, metric=np.eye(k))
    C3, D3 = ocb.lloyd_max(d, k, N, 1, 20000, 2, 6, metric=3.0 * np.eye(k))
    assert np.array_equal(C, C1) and D1 == pytest.approx(D, rel=1e-12)
    assert np.array_equal(C, C3) and D3 == pytest.approx(3.0 * D, rel=1e-12)


# ------------------------------------------------ sub-linear encoders (App. F) ---
def _tiny_setup(d=16, k=4, N=32, L=4, n=40, seed=2):
    C = ocb.multishell_codebook(d, k, L, N // L)
    R = oracle_rotation(d)
    x = np.random.default_rng(seed).standard_normal((n, d))
    return C, R, x


def test_radius_first_single_shell_is_exhaustive():
    """App. F Stage 1 with one shell searches every codeword: the indices are
    the exhaustive encoder's (Eq. encode)."""
    d, k, N = 64, 4, 64
    C, _ = oracle_codebook(d, k, N, M=20000)
    R = oracle_rotation(d)
    x = np.random.default_rng(4).standard_normal((300, d))
    i0, h0 = occ.encode(x, R, C)
    i1, h1, shell = osl.encode_radius_first(x, R, C, 1)
    assert np.array_equal(i0, i1) and np.array_equal(h0, h1) and (shell == 0).all()


def test_radius_first_brute_force_tiny():
    """App. F Stage 1 written out with plain loops on tiny inputs: the shell
    is the one whose Eq. multishell radius is nearest to ||y^(m)|| (lower
    shell on ties), the codeword the nearest of that shell, the index
    l* M_a + n."""
    d, k, N, L = 16, 4, 32, 4
    C, R, x = _tiny_setup(d, k, N, L)
    Ma = N // L
    beta = k / (k + 2) * (d - k - 2) / 2 + 1
    r = [math.sqrt(betaincinv(k / 2, beta, (l + 0.5) / L)) for l in range(L)]
    idx, _, _ = osl.encode_radius_first(x, R, C, L)
    for v in range(x.shape[0]):
        nu = math.sqrt(sum(t * t for t in x[v]))
        y = [sum(R[i, j] * x[v, j] for j in range(d)) / nu for i in range(d)]
        for m in range(d // k):
            b = y[m * k:(m + 1) * k]
            rho = math.sqrt(sum(t * t for t in b))
            best_l = min(range(L), key=lambda l: (abs(rho - r[l]), l))
            dist = [sum((b[i] - C[best_l * Ma + n, i]) ** 2 for i in range(k)) for n in range(Ma)]
            n_star = min(range(Ma), key=lambda n: (dist[n], n))
            assert idx[v, m] == best_l * Ma + n_star


def test_radius_first_recovers_codewords_on_their_shell():
    """A block equal to codeword r_l u_n of the construction C(L, M_a) is
    encoded as l M_a + n (App. F: the index is the affine pair offset)."""
    d, k, L, Ma = 64, 4, 8, 16
    C = ocb.multishell_codebook(d, k, L, Ma)
    idx, shell = osl.search_blocks(C, C, L, osl.shell_radii(d, k, L))
    assert np.array_equal(idx, np.arange(L * Ma))
    assert np.array_equal(shell, np.arange(L * Ma) // Ma)


def test_hierarchical_full_list_is_radius_first():
    """App. F Stage 2 with T = K searches every child of the shell: the same
    indices as Stage 1 alone; a shorter list never finds a nearer codeword."""
    d, k, N, L = 64, 8, 256, 8
    C, _ = ocb.lloyd_max(d, k, N, 1, 20000, 1, 10, init="multishell", shells=L)
    R = oracle_rotation(d)
    x = np.random.default_rng(6).standard_normal((120, d))
    i1, _, _ = osl.encode_radius_first(x, R, C, L)
    i_full, _ = osl.encode_hierarchical(x, R, C, L, K=4, T=4)
    assert np.array_equal(i1, i_full)
    i_t1, _ = osl.encode_hierarchical(x, R, C, L, K=4, T=1)
    y = occ.rotate_normalise(x, R, occ.norms(x)[0]).reshape(-1, k)
    d1 = ((y - C[i1.reshape(-1)]) ** 2).sum(1)
    dt = ((y - C[i_t1.reshape(-1)]) ** 2).sum(1)
    assert (dt >= d1 - 1e-15).all()
