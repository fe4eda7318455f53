"""Shared Haar rotation and radial-angular codebook construction (oracle side).

Test infrastructure only.  Follows the paper step by step:

* Haar rotation: the shared orthogonal matrix of Sec. 3 (Fig. 1 caption,
  Sec. 3.1).  Generated as the Q factor of a d x d standard-normal matrix with
  the signs of R's diagonal folded into Q, which makes Q Haar distributed
  (Mezzadri 2007).  Normals come from the Philox stream (``philox``).
* Spherical-Beta source f_{d,k} (Lemma 1): the first k coordinates of a
  uniform point on S^{d-1}, sampled as a normalised d-dim Gaussian.
* Beta-quantile radii (Eq. radii_main, closed form Eq. radii_k2 at k = 2).
* Direction sets (Sec. 3.3 "Directions"; App. E Eq. fib_sphere_3d).
* Multi-restart Lloyd-Max polish (App. A, codebook-construction table).
* Alternative starting codebooks for the same polish: the large-d single
  shell (App. D) and the multi-shell C(S, M_a) with its factor-pair search
  (App. E Eq. multishell).  The full-vector code k = d needs nothing special:
  the source is then the whole unit vector and Eq. radii_main stays defined.

Readings where the paper leaves freedom (restated in the design notes):
k = 1 directions alternate +1/-1 with n; each restart rotates the initial
codebook by its own Haar k x k matrix; an empty cell is refilled by splitting
the occupied cell with the largest within-cell squared error (donor moves by
-delta, the empty codeword is placed at donor + delta, delta a random
direction of length 1e-2 times the donor cell's rms radius); D(C) is the
training MSE after one final assignment; training samples are one k-block per
normalised Gaussian; a multi-shell "fresh" direction set is the next M_a
points of the same sequence (at k = 3 only the azimuth continues, the
latitude bands restart per shell), codewords shell-major.
"""
import math

import numpy as np
from scipy.special import betaincinv, ndtri

from . import philox

GOLDEN = (1.0 + math.sqrt(5.0)) / 2.0


# ---------------------------------------------------------------- rotation ---
def haar_from_normals(g):
    """Haar-distributed orthogonal Q from a square standard-normal matrix g."""
    q, r = np.linalg.qr(g)
    s = np.sign(np.diag(r))
    s[s == 0] = 1.0
    return q * s[None, :]


def haar_rotation(d, seed):
    """Shared rotation Pi (d x d, float64), y = Pi x (row-major, Sec. 3.1)."""
    g = philox.normals(seed, philox.TAG_ROTATION, 0, d * d).reshape(d, d)
    return haar_from_normals(g)


# ------------------------------------------------------------------ source ---
def sample_source(d, k, count, seed, tag=philox.TAG_TRAIN, start=0):
    """``count`` draws of f_{d,k} (Lemma 1): first k coords of U ~ Unif(S^{d-1}).

    Sample s uses normals ``(start + s) * d .. + d - 1`` of stream (seed, tag).
    """
    out = np.empty((count, k))
    step = max(1, (1 << 16) // d)
    for s in range(0, count, step):
        c = min(step, count - s)
        g = philox.normals(seed, tag, (start + s) * d, c * d).reshape(c, d)
        out[s:s + c] = g[:, :k] / np.sqrt((g * g).sum(axis=1, keepdims=True))
    return out


# ------------------------------------------------------------------- radii ---
def beta_dk(d, k):
    """beta_{d,k} = k/(k+2) * (d-k-2)/2 + 1 (Eq. radii_main)."""
    return k / (k + 2.0) * (d - k - 2.0) / 2.0 + 1.0


def radii(d, k, N):
    """Beta-quantile radii r_n, n = 1..N (Eq. radii_main; Eq. radii_k2 at k=2)."""
    q = (np.arange(1, N + 1) - 0.5) / N
    if k == 2:
        return np.sqrt(1.0 - (1.0 - q) ** (4.0 / d))
    return np.sqrt(betaincinv(k / 2.0, beta_dk(d, k), q))


# -------------------------------------------------------------- directions ---
def roberts_phi(k):
    """Positive root of phi^(k+1) = phi + 1 (Sec. 3.3, k >= 4), by bisection."""
    lo, hi = 1.0, 2.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mid ** (k + 1) - mid - 1.0 > 0:
            hi = mid
        else:
            lo = mid
    return 0.5 * (lo + hi)


def directions(k, N, offset=0):
    """Quasi-uniform unit directions u_n on S^{k-1}, n = offset+1 .. offset+N
    (Sec. 3.3).  ``offset`` > 0 continues the sequence, which is how each shell
    of the multi-shell codebook gets a fresh set (App. E); at k = 3 the
    equal-area latitude uses the local index 1..N and only the golden-angle
    azimuth continues."""
    n = np.arange(offset + 1, offset + N + 1, dtype=np.float64)
    if k == 1:
        return np.where(n % 2 == 1, 1.0, -1.0)[:, None]
    if k == 2:
        theta = 2.0 * np.pi * (n - 1.0) * (1.0 - 1.0 / GOLDEN)
        return np.stack([np.cos(theta), np.sin(theta)], axis=1)
    if k == 3:
        z = 1.0 - (2.0 * (n - offset) - 1.0) / N
        theta = 2.0 * np.pi * (n - 1.0) * (1.0 - 1.0 / GOLDEN)
        rho = np.sqrt(1.0 - z * z)
        return np.stack([rho * np.cos(theta), rho * np.sin(theta), z], axis=1)
    g = ndtri(kronecker_points(k, N, offset))
    return g / np.linalg.norm(g, axis=1, keepdims=True)


def kronecker_points(k, N, offset=0):
    """Roberts-Kronecker points xi_{n,j} = {(n - 1/2) phi_k^(-j)}, j = 1..k, in
    the unit cube (Sec. 3.3, k >= 4), n = offset+1 .. offset+N; the k >= 4
    directions are Phi^-1(xi_n) projected onto the sphere."""
    n = np.arange(offset + 1, offset + N + 1, dtype=np.float64)
    phi = roberts_phi(k)
    j = np.arange(1, k + 1, dtype=np.float64)
    return np.mod((n[:, None] - 0.5) * phi ** (-j[None, :]), 1.0)


def initial_codebook(d, k, N):
    """C^(0) = {r_n u_n} (App. A table, lines 1-8)."""
    return radii(d, k, N)[:, None] * directions(k, N)


def single_shell_codebook(d, k, N):
    """Large-d shortcut (App. D; App. A table footnote): every radius is the
    typical radius sqrt(k/d), the directions are unchanged."""
    return math.sqrt(k / d) * directions(k, N)


def multishell_codebook(d, k, S, Ma):
    """C(S, M_a) of App. E Eq. multishell: S shells at the Beta quantiles
    q_s = (s - 1/2)/S, each carrying a fresh M_a-point direction set."""
    r = radii(d, k, S)
    return np.concatenate([r[s] * directions(k, Ma, offset=s * Ma) for s in range(S)])


def choose_multishell(d, k, N, x):
    """Enumerate every factor pair S * M_a = N (App. E) and keep the C(S, M_a)
    with the lowest training MSE on x (ties: the smaller S).  Returns (S, C)."""
    best = None
    for S in range(1, N + 1):
        if N % S:
            continue
        c = multishell_codebook(d, k, S, N // S)
        _, e = _nearest_chunked(x, c)
        m = float(e.mean())
        if best is None or m < best[0]:
            best = (m, S, c)
    return best[1], best[2]


def starting_codebook(d, k, N, init, x, shells=0):
    """The codebook Lloyd starts from, and its number of radial shells:
    "beta" (N Beta-quantile shells), "shell" (the large-d single shell) or
    "multishell" (C(shells, N / shells) when ``shells`` > 0, e.g. the sqrt(N)
    shells of the radius-first encoder of App. F; else the best factor pair
    on the training sample x)."""
    if init == "beta":
        return initial_codebook(d, k, N), N
    if init == "shell":
        return single_shell_codebook(d, k, N), 1
    if init == "multishell":
        if shells > 0:
            if N % shells:
                raise ValueError("shells must divide N")
            return multishell_codebook(d, k, shells, N // shells), shells
        S, c = choose_multishell(d, k, N, x)
        return c, S
    raise ValueError(f"unknown init {init!r}")


# ------------------------------------------------------------------- Lloyd ---
def nearest(x, c, metric=None):
    """Index of the nearest codeword for each row of x (ties: lowest index) and
    the squared distance ||x - c_j||^2, by brute force over all codewords.
    With a k x k ``metric`` M the distance is (x - c)^T M (x - c) (the
    task-weighted / Mahalanobis objective of Sec. 3, Eq. lattn discussion)."""
    dist = np.zeros((x.shape[0], c.shape[0]))
    if metric is None:
        for i in range(x.shape[1]):
            dist += (x[:, i:i + 1] - c[None, :, i]) ** 2
    else:
        for i in range(x.shape[1]):
            for j in range(x.shape[1]):
                dist += (x[:, i:i + 1] - c[None, :, i]) * metric[i, j] * (x[:, j:j + 1] - c[None, :, j])
    a = dist.argmin(axis=1)
    return a, dist[np.arange(x.shape[0]), a]


def _nearest_chunked(x, c, chunk=1024, metric=None):
    a = np.empty(x.shape[0], dtype=np.int64)
    e = np.empty(x.shape[0], dtype=np.float64)
    for s in range(0, x.shape[0], chunk):
        a[s:s + chunk], e[s:s + chunk] = nearest(x[s:s + chunk], c, metric)
    return a, e


def lloyd_round(x, c, seed, repair_events, metric=None):
    """One Lloyd-Max round on training samples x (App. A table, lines 13-18):
    assign every sample to its nearest codeword, move each occupied codeword to
    its cell mean, then refill each empty cell (in index order) by splitting
    the occupied cell of >= 2 members with the largest within-cell squared
    error: the donor moves by -delta and the empty codeword is placed at
    donor + delta, delta = 1e-2 x the donor's rms error x a unit direction
    from Philox normals (seed, repair tag) numbered by ``repair_events``; the
    donor's error is halved and half its members are counted to the new
    cell.  Returns (new codebook, updated repair count)."""
    c = c.copy()
    N, k = c.shape
    a, _ = _nearest_chunked(x, c, metric=metric)
    counts = np.bincount(a, minlength=N)
    occ = counts > 0
    for i in range(k):  # centroid of each occupied cell
        sums = np.bincount(a, weights=x[:, i], minlength=N)
        c[occ, i] = sums[occ] / counts[occ]
    diff = x - c[a]
    err = (diff ** 2).sum(axis=1) if metric is None else ((diff @ metric) * diff).sum(axis=1)
    sse = np.bincount(a, weights=err, minlength=N)
    for e in range(N):
        if counts[e] > 0:
            continue
        cand = np.where(counts >= 2, sse, -1.0)
        donor = int(np.argmax(cand))
        if cand[donor] < 0:
            break
        g = philox.normals(seed, philox.TAG_REPAIR, repair_events * k, k)
        repair_events += 1
        gn = np.linalg.norm(g)
        u = g / gn if gn > 0 else np.eye(k)[0]
        delta = 1e-2 * math.sqrt(sse[donor] / counts[donor]) * u
        c[e] = c[donor] + delta
        c[donor] = c[donor] - delta
        sse[donor] *= 0.5
        half = counts[donor] // 2
        counts[e] = half
        counts[donor] -= half
    return c, repair_events


def lloyd_max(d, k, N, seed, M, restarts, iters, return_trace=False, init="beta",
              return_shells=False, shells=0, metric=None):
    """Multi-restart Lloyd-Max refinement (App. A table, lines 9-20).

    Returns (C*, D*) with D* the per-block training MSE of the kept codebook
    (then the trace of D(C) per restart if ``return_trace``, then the number
    of radial shells of the starting codebook if ``return_shells``).  With a
    symmetric positive definite k x k ``metric`` M every squared error is
    (x - c)^T M (x - c): assignments, the repair donor's error and D(C) use
    it, and the cell mean stays the optimal centroid (the gradient of the
    cell's error, -2 M sum (x - c), vanishes there).
    """
    if metric is not None:
        metric = np.asarray(metric, dtype=np.float64)
    x = sample_source(d, k, M, seed, philox.TAG_TRAIN)
    c0, shells = starting_codebook(d, k, N, init, x, shells)
    best_c, best_d = c0.copy(), np.inf
    repair_events = 0
    trace = []
    for j in range(restarts):
        omega = haar_from_normals(
            philox.normals(seed, philox.TAG_RESTART, j * k * k, k * k).reshape(k, k))
        c = c0 @ omega.T  # c_n <- Omega_j c_n
        for _ in range(iters):
            c, repair_events = lloyd_round(x, c, seed, repair_events, metric)
        _, err = _nearest_chunked(x, c, metric=metric)
        dj = float(err.mean())
        trace.append(dj)
        if dj < best_d:
            best_c, best_d = c.copy(), dj
    out = (best_c, best_d)
    if return_trace:
        out += (trace,)
    if return_shells:
        out += (shells,)
    return out


def build_codebook(d, k, N, seed, M=None, restarts=4, iters=25, init="beta", shells=0,
                   metric=None):
    """FibQuant codebook for (d, k, N); M defaults to 30 N (Sec. 5.1)."""
    if M is None:
        M = 30 * N
    return lloyd_max(d, k, N, seed, M, restarts, iters, init=init, shells=shells, metric=metric)


def mse_on(c, d, k, count, seed, tag=philox.TAG_HELDOUT):
    """Per-block MSE of codebook c on ``count`` fresh f_{d,k} samples (L_mse / (d/k))."""
    x = sample_source(d, k, count, seed, tag)
    _, e = _nearest_chunked(x, c)
    return float(e.mean())


def nmse_db(block_mse, d, k):
    """Per-vector NMSE in dB: (d/k) block MSE against E||unit vector||^2 = 1."""
    return 10.0 * math.log10(block_mse * d / k)
