"""Sub-linear encoders for large codebooks (oracle side, float64).

Test infrastructure only.  App. F ("hierarchical list decoding") describes two
ways to search a multi-shell codebook (App. E Eq. multishell) in fewer than N
inner products per k-block, with the bitstream and the decoder unchanged:

* Stage 1, radius-first: with L shells of M_a = N / L codewords each, stored
  shell-major (shell l holds indices l M_a .. (l + 1) M_a - 1, radius r_l),
  block m of the rotated unit vector y picks the shell whose radius is nearest
  to rho = ||y^(m)||, then the nearest codeword of that shell alone; the
  index is l* M_a + n.  O(L + N / L) work instead of O(N).
* Stage 2, hierarchical direction code: the M_a codewords of a shell are
  grouped into K parents; the block's direction is compared with the parents'
  mean directions, the children of the best T parents form a candidate list,
  and the list is searched exhaustively.  T = K is the exhaustive shell search.

Readings where the paper leaves freedom (restated in the design notes): the
shell radii are the construction radii of Eq. multishell, r_l =
sqrt(BetaInv((l - 1/2) / L; k/2, beta_dk)), also after the Lloyd polish has
moved the codewords; ties go to the lower shell and to the lower index; a
zero block (rho = 0) takes shell 0.  Stage 2's parents come from spherical
k-means on the shell's codeword directions, started from every (M_a / K)-th
codeword and run a fixed number of rounds (a group that empties keeps its
previous mean); the top-T parents are ranked by inner product, ties to the
lower parent.
"""
import numpy as np

from . import codebook as ocb
from . import codec as occ


def shell_radii(d, k, L):
    """r_l of App. E Eq. multishell, l = 1..L (the Beta quantiles at (l - 1/2)/L)."""
    return ocb.radii(d, k, L)


def nearest_shell(rho, r):
    """argmin_l |rho - r_l| for each rho (App. F Stage 1, step 1), lower l on ties."""
    return np.abs(np.asarray(rho)[..., None] - r[None, :]).argmin(axis=-1)


def search_blocks(blocks, C, L, r):
    """App. F Stage 1 on k-blocks [nb, k]: (index l* M_a + n, shell l*) per block."""
    N, k = C.shape
    Ma = N // L
    rho = np.sqrt((blocks * blocks).sum(axis=1))
    shell = nearest_shell(rho, r)
    idx = np.empty(blocks.shape[0], dtype=np.int64)
    for l in range(L):
        sel = shell == l
        if not sel.any():
            continue
        cs = C[l * Ma:(l + 1) * Ma]
        b = blocks[sel]
        D = np.zeros((b.shape[0], Ma))
        for i in range(k):
            D += (b[:, i:i + 1] - cs[None, :, i]) ** 2
        idx[sel] = l * Ma + D.argmin(axis=1)
    return idx, shell


def encode_radius_first(x, Pi, C, L):
    """Stage 1 encoder: (indices [n, d/k], fp16 headers [n], chosen shells
    [n, d/k]).  C is shell-major with L shells of N / L codewords; the shell
    radii follow the spherical-Beta law of the head dimension d."""
    x = np.asarray(x, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    N, k = C.shape
    if N % L:
        raise ValueError("L must divide N")
    n, d = x.shape
    nu, h = occ.norms(x)
    y = occ.rotate_normalise(x, Pi, nu)
    idx, shell = search_blocks(y.reshape(-1, k), C, L, shell_radii(d, k, L))
    idx, shell = idx.reshape(n, d // k), shell.reshape(n, d // k)
    zero = nu == 0
    idx[zero] = 0
    shell[zero] = 0
    h[zero] = np.float16(0.0)
    return idx, h, shell


def parent_groups(U, K, rounds=10):
    """Spherical k-means of the unit directions U [M_a, k] into K parents
    (App. F Stage 2): returns (group of each codeword [M_a], parent mean
    directions [K, k])."""
    Ma = U.shape[0]
    mu = U[:: Ma // K][:K].copy()
    g = np.zeros(Ma, dtype=np.int64)
    for _ in range(rounds):
        g = (U @ mu.T).argmax(axis=1)
        for j in range(K):
            m = U[g == j].sum(axis=0)
            n = np.linalg.norm(m)
            if n > 0:
                mu[j] = m / n
    g = (U @ mu.T).argmax(axis=1)
    return g, mu


def encode_list(y_blocks, cs, groups, mu, T):
    """Stage 2 search of one shell: for each block (rows of y_blocks), the
    children of the T parents with the largest <v, mu_j> (v = y / ||y||) are
    searched exhaustively; returns the local index of the nearest of them."""
    nb = y_blocks.shape[0]
    rho = np.linalg.norm(y_blocks, axis=1)
    v = y_blocks / np.where(rho > 0, rho, 1.0)[:, None]
    score = v @ mu.T
    order = np.argsort(-score, axis=1, kind="stable")[:, :T]
    out = np.empty(nb, dtype=np.int64)
    for b in range(nb):
        cand = np.flatnonzero(np.isin(groups, order[b]))
        dist = ((y_blocks[b][None, :] - cs[cand]) ** 2).sum(axis=1)
        out[b] = cand[dist.argmin()]
    return out


def parent_tables(C, L, K, rounds=10):
    """Stage 2 tables of a shell-major codebook: (mu [L, K, k] parent mean
    directions, groups [N] parent of each codeword within its shell)."""
    C = np.asarray(C, dtype=np.float64)
    N, k = C.shape
    Ma = N // L
    mu = np.empty((L, K, k))
    groups = np.empty(N, dtype=np.int64)
    for l in range(L):
        cs = C[l * Ma:(l + 1) * Ma]
        U = cs / np.linalg.norm(cs, axis=1, keepdims=True)
        groups[l * Ma:(l + 1) * Ma], mu[l] = parent_groups(U, K, rounds)
    return mu, groups


def encode_hierarchical_tables(x, Pi, C, L, mu, groups, T):
    """Stages 1 + 2 with given parent tables: (indices [n, d/k], fp16 headers)."""
    x = np.asarray(x, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    N, k = C.shape
    Ma = N // L
    d = x.shape[1]
    r = shell_radii(d, k, L)
    nu, h = occ.norms(x)
    y = occ.rotate_normalise(x, Pi, nu)
    blocks = y.reshape(-1, k)
    shell = nearest_shell(np.linalg.norm(blocks, axis=1), r)
    idx = np.zeros(blocks.shape[0], dtype=np.int64)
    for l in range(L):
        sel = np.flatnonzero(shell == l)
        if sel.size == 0:
            continue
        cs = C[l * Ma:(l + 1) * Ma]
        idx[sel] = l * Ma + encode_list(blocks[sel], cs, groups[l * Ma:(l + 1) * Ma], mu[l], T)
    idx = idx.reshape(x.shape[0], d // k)
    zero = nu == 0
    idx[zero] = 0
    h[zero] = np.float16(0.0)
    return idx, h


def encode_hierarchical(x, Pi, C, L, K, T, rounds=10):
    """Stages 1 + 2 composed (App. F "Composition"): nearest shell by radius,
    then list decoding inside it.  Returns (indices, fp16 headers)."""
    mu, groups = parent_tables(C, L, K, rounds)
    return encode_hierarchical_tables(x, Pi, C, L, mu, groups, T)
