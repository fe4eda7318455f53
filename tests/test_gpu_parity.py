"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Inputs are seeded synthetic caches (paper_2605_11478_amd.workloads) with the
workloads' dtypes, element laws, (d, k, N) and group layout, shrunk in layers
and tokens so the float64 oracle finishes in seconds while still spanning
several tiles and a ragged tail.  Bars: indices exact except inside the 1e-6
near-tie window, payload bytes and fp16 norm bits exact, reconstructions
within 1e-5 max(1, nu), attention within 2e-3 relative l2 per head.
"""
import math

import numpy as np
import pytest
import torch

import paper_2605_11478_amd as fq
from paper_2605_11478_amd import workloads as W
from oracle import codebook as ocb
from oracle import codec as occ
from oracle import sublinear as osl

from _fixtures import oracle_rotation, quick_codebook
import gpu_helpers as gh

pytestmark = pytest.mark.gpu

CASES = [(name, k, N) for name, wl in W.WORKLOADS.items() for (k, N) in wl.rates]
SMALL = {  # (layers, T) used for the reduced-size parity runs
    "tiny": (1, 4096), "gpt2": (2, 333), "tinyllama": (1, 203), "long32k": (1, 450),
    "stress": (1, 70),
}


def _setup(wl, k, N, dev):
    R = oracle_rotation(wl.d)
    C = quick_codebook(wl.d, k, N)
    return R, C, torch.from_numpy(R.copy()).to(dev), torch.from_numpy(C.copy()).to(dev)


def _say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("name,k,N", CASES)
def test_encode_decode_attention_parity(name, k, N, device):
    wl = W.WORKLOADS[name]
    L, T = SMALL[name]
    _say(f"[parity] {name} k={k} N={N} layers={L} T={T}")
    R, C, Rd, Cd = _setup(wl, k, N, device)
    kc = W.make_cache(wl, "k", "cpu", T=T, layers=L)
    vc = W.make_cache(wl, "v", "cpu", T=T, layers=L)
    q = W.group_view_query(W.make_query(wl, "cpu", layers=L), wl)
    n_g = q.shape[0]
    d = wl.d
    if name == "stress":  # keep the float64 oracle (N = 4096) to seconds
        kc, vc, q = kc[:, :, :2], vc[:, :, :2], q.reshape(L, wl.batch, wl.kv_heads, wl.G, d)[:, :, :2]
        q = q.reshape(-1, wl.G, d)
        n_g = q.shape[0]
    kx = kc.reshape(-1, d).contiguous()
    vx = vc.reshape(-1, d).contiguous()

    # encode on the device, parity against the oracle
    kp, kn = fq.encode(kx.to(device), k, N, Rd, Cd)
    vp, vn = fq.encode(vx.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, k_idx, k_h = gh.check_encode(gh.host_f64(kx), R, C, N, kp, kn)
    ne2, nt2, v_idx, v_h = gh.check_encode(gh.host_f64(vx), R, C, N, vp, vn)
    _say(f"  encode: {ne + ne2} exact indices, {nt + nt2} accepted near-ties")

    # decode: device decoder on the oracle's payload vs the oracle decoder
    k_pay = occ.pack(k_idx, N)
    v_pay = occ.pack(v_idx, N)
    k_nb = occ.fp16_bits(k_h)
    v_nb = occ.fp16_bits(v_h)
    pd = torch.from_numpy(k_pay).to(device)
    nd = torch.from_numpy(k_nb.view(np.int16)).to(device)
    xh = fq.decode(pd, nd, d, k, N, Rd, Cd)
    ref = occ.decode(k_idx, k_h, R.astype(np.float64), C.astype(np.float64))
    gh.check_recon(xh.cpu().numpy(), ref, k_h)
    ids = torch.randint(0, pd.shape[0], (777,), generator=torch.Generator().manual_seed(1))
    xs = fq.decode(pd, nd, d, k, N, Rd, Cd, token_ids=ids.to(device))
    assert torch.equal(xs.cpu(), xh.cpu()[ids]), "random-access rows differ from the range decode"

    # attention: device kernel on the oracle's payload vs naive oracle attention
    P = k_pay.shape[1]
    kpg = torch.from_numpy(k_pay.reshape(n_g, T, P)).to(device)
    vpg = torch.from_numpy(v_pay.reshape(n_g, T, P)).to(device)
    kng = torch.from_numpy(k_nb.view(np.int16).reshape(n_g, T)).to(device)
    vng = torch.from_numpy(v_nb.view(np.int16).reshape(n_g, T)).to(device)
    o = fq.attn_decode(q.to(device), kpg, kng, vpg, vng, T, k, N, Rd, Cd)
    o_ref = gh.oracle_group_attention(gh.host_f64(q), k_pay.reshape(n_g, T, P),
                                      k_nb.reshape(n_g, T), v_pay.reshape(n_g, T, P),
                                      v_nb.reshape(n_g, T), R, C, N, T)
    rel = gh.check_attention(o.cpu().numpy(), o_ref)
    _say(f"  attention: max rel l2 {rel:.2e}")

    # end to end: the device's own payload through the device attention
    o2 = fq.attn_decode(q.to(device), kp.reshape(n_g, T, P), kn.reshape(n_g, T),
                        vp.reshape(n_g, T, P), vn.reshape(n_g, T), T, k, N, Rd, Cd)
    gh.check_attention(o2.cpu().numpy(), o_ref)


@pytest.mark.parametrize("dtype", [torch.float32, torch.float16, torch.bfloat16])
def test_encode_edge_cases(dtype, device):
    """Zero vectors, norms at binary16 rounding midpoints, overflow, subnormal
    headers, strided rows and a ragged count (not a multiple of 256)."""
    d, k, N = 64, 4, 256
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(7)
    x = torch.randn(517, 2 * d, generator=g).to(dtype)
    x[3] = 0
    specials = [1.0 + 2 ** -11, 1.0 + 3 * 2 ** -11, 65504.0, 65519.0, 65520.0, 3e5,
                2.0 ** -24, 3 * 2.0 ** -25, 2.0 ** -26]
    for i, v in enumerate(specials):
        x[10 + i] = 0
        x[10 + i, 5] = v
    if dtype != torch.float32:  # keep finite in the narrow types
        x[10:10 + len(specials)] = x[10:10 + len(specials)].clamp(-6e4, 6e4)
    xs = x[:, :d]  # strided rows (stride 2d)
    xd = x.to(device)[:, :d]
    assert xd.stride(0) == 2 * d
    _say(f"[edge] encode dtype={dtype}")
    p, nrm = fq.encode(xd, k, N, Rd, Cd)
    torch.cuda.synchronize()
    gh.check_encode(gh.host_f64(xs), R, C, N, p, nrm)
    assert int(gh.bits_u16(nrm)[3]) == 0 and not p.cpu().numpy()[3].any()
    # determinism: a second run gives the same bytes
    p2, n2 = fq.encode(xd, k, N, Rd, Cd)
    assert torch.equal(p, p2) and torch.equal(nrm, n2)


@pytest.mark.parametrize("N,fp16_cb", [(16, True), (16, False), (64, True), (64, False)])
def test_encode_bf16_k8_screen_path(N, fp16_cb, device):
    """bf16 rows at d = 64, k = 8 (the matrix-core screen with its float64
    near-tie and out-of-range paths): norms spread over many decades, a zero
    row, a header above the binary16 range, a binary16-subnormal header, rows
    whose squared sums leave the float32 range, strided rows, a ragged count,
    and codebooks with and without exact binary16 entries."""
    d, k = 64, 8
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    if fp16_cb:
        C = C.astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(11 + N)
    n = 4099
    x = torch.randn(n, 2 * d, generator=g) * torch.exp(2 * torch.randn(n, 1, generator=g))
    x[5] = 0
    x[6, :d] = 0
    x[6, 3] = 3e5                                       # header overflows to +inf
    x[7, :d] = 1e30                                     # sum of squares above 2^100
    x[8, :d] = 1e-30 * torch.randn(d, generator=g)      # below 2^-100
    x[9, :d] = 0
    x[9, 17] = 2.0 ** -20                               # binary16-subnormal header
    x = x.to(torch.bfloat16)
    xs = x[:, :d]
    xd = x.to(device)[:, :d]
    assert xd.stride(0) == 2 * d
    _say(f"[edge] bf16 k=8 screen path N={N} fp16 codebook={fp16_cb}")
    p, nrm = fq.encode(xd, k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(xs), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")
    p2, n2 = fq.encode(xd, k, N, Rd, Cd)
    assert torch.equal(p, p2) and torch.equal(nrm, n2)


@pytest.mark.parametrize("N", [16, 64])
def test_encode_bf16_k8_many_out_of_range_rows(N, device):
    """Tiles with many rows whose squared sums leave the float32 range (every
    block of such a row is redone in float64): a 32-row tile with 16 of them,
    more than the encoder's per-wavefront queue of deferred blocks holds, a
    tile with 4 (exactly a full queue) and scattered single rows, among
    ordinary rows and near ties."""
    d, k = 64, 8
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(23 + N)
    n = 1000
    x = torch.randn(n, d, generator=g) * torch.exp(torch.randn(n, 1, generator=g))
    for r in list(range(32, 48)) + list(range(64, 68)) + [101, 333, 517, 999]:
        x[r] = (1e30 if r % 2 else 1e-30) * torch.randn(d, generator=g)
    x = x.to(torch.bfloat16)
    _say(f"[edge] bf16 k=8 many out-of-range rows N={N}")
    p, nrm = fq.encode(x.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(x), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")


@pytest.mark.parametrize("N", [16, 64])
def test_encode_bf16_k8_near_midpoints(N, device):
    """Rows built so that seven of the eight blocks of y sit at the midpoint of
    a codeword and its nearest neighbour (the eighth block makes |y| = 1), then
    rounded to bf16: thousands of blocks fall within the screen's certification
    margin or just above it, and every index must still be the float64 argmin
    (up to the 1e-6 near-tie window)."""
    d, k = 64, 8
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    C64 = C.astype(np.float64)
    D2 = ((C64[:, None, :] - C64[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(D2, np.inf)
    nbr = D2.argmin(1)
    rng = np.random.default_rng(100 + N)
    n = 8192
    a = rng.integers(0, N, size=(n, 7))
    mid = 0.5 * (C64[a] + C64[nbr[a]])                     # [n, 7, k]
    rest = 1.0 - (mid ** 2).sum(axis=(1, 2))
    assert np.all(rest > 0)
    last = rng.standard_normal((n, k))
    last *= (np.sqrt(rest) / np.linalg.norm(last, axis=1))[:, None]
    y = np.concatenate([mid.reshape(n, 7 * k), last], axis=1)
    nu = np.exp(rng.uniform(-3.0, 3.0, size=(n, 1)))
    x = (nu * (y @ R.astype(np.float64))).astype(np.float32)  # Pi x = nu y, Pi = R
    xs = torch.from_numpy(x).to(torch.bfloat16)
    # the oracle's own margins on these rows: how many blocks are close calls
    _, _, D = occ.encode(gh.host_f64(xs), R.astype(np.float64), C64, return_distances=True)
    Dsort = np.sort(D, axis=-1)
    close = int(((Dsort[..., 1] - Dsort[..., 0]) <= 1e-3 * Dsort[..., 1]).sum())
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    _say(f"[edge] bf16 k=8 near midpoints N={N}: {close} blocks within 1e-3 relative")
    assert close > 1000
    p, nrm = fq.encode(xs.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(xs), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")


@pytest.mark.parametrize("k,N,dtype,fp16_cb", [
    (4, 256, torch.bfloat16, True), (4, 256, torch.float16, False), (4, 64, torch.bfloat16, False),
    (4, 64, torch.float16, True), (4, 16, torch.float16, True), (2, 64, torch.bfloat16, True),
    (2, 64, torch.float16, False), (2, 16, torch.bfloat16, False), (2, 256, torch.float16, True)])
def test_encode_k4_k2_screen_path(k, N, dtype, fp16_cb, device):
    """bf16 / fp16 rows at d = 64 with k = 4 or 2 (the matrix-core screen with
    its float64 near-tie and out-of-range paths): norms spread over many
    decades, a zero row, a header above the binary16 range, a
    binary16-subnormal header, sums of squares outside [2^-100, 2^100]
    (bf16), strided rows, a ragged count, codebooks with and without exact
    binary16 entries."""
    d = 64
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    if fp16_cb:
        C = C.astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(31 + 7 * k + N)
    n = 4099
    x = torch.randn(n, 2 * d, generator=g) * torch.exp(2 * torch.randn(n, 1, generator=g))
    if dtype == torch.float16:
        x = x.clamp(-6e4, 6e4)
    x[5] = 0
    x[6, :d] = 0
    x[6, 3] = 3e5 if dtype == torch.bfloat16 else 6e4
    if dtype == torch.float16:
        x[6, 4] = 6e4                                   # header 84853 overflows to +inf
    if dtype == torch.bfloat16:
        x[7, :d] = 1e30                                 # sum of squares above 2^100
        x[8, :d] = 1e-30 * torch.randn(d, generator=g)  # below 2^-100
    else:
        x[7, :d] = 2.0 ** -24 * torch.randint(-3, 4, (d,), generator=g)  # binary16 subnormals
    x[9, :d] = 0
    x[9, 17] = 2.0 ** -20                               # binary16-subnormal header
    x = x.to(dtype)
    xs = x[:, :d]
    xd = x.to(device)[:, :d]
    assert xd.stride(0) == 2 * d
    _say(f"[edge] k={k} N={N} {dtype} screen path fp16 codebook={fp16_cb}")
    p, nrm = fq.encode(xd, k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(xs), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")
    p2, n2 = fq.encode(xd, k, N, Rd, Cd)
    assert torch.equal(p, p2) and torch.equal(nrm, n2)


@pytest.mark.parametrize("k,N,dtype", [(4, 256, torch.bfloat16), (4, 256, torch.float16),
                                       (2, 64, torch.bfloat16), (2, 16, torch.float16)])
def test_encode_k4_k2_near_midpoints(k, N, dtype, device):
    """Rows whose first half (k = 4) or third (k = 2) of the blocks sit at the
    midpoint of a codeword and its nearest neighbour (the other blocks random,
    scaled so that |y| = 1), rounded to the cache dtype: many close calls for
    the k = 4 / k = 2 screen's margin; every index must be the float64 argmin
    (1e-6 window)."""
    d = 64
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    C64 = C.astype(np.float64)
    D2 = ((C64[:, None, :] - C64[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(D2, np.inf)
    nbr = D2.argmin(1)
    rng = np.random.default_rng(200 + 7 * k + N)
    n, nb = 8192, d // k
    m = nb // 2 if k == 4 else nb // 3
    a = rng.integers(0, N, size=(n, m))
    mid = 0.5 * (C64[a] + C64[nbr[a]])                     # [n, m, k]
    rest = 1.0 - (mid ** 2).sum(axis=(1, 2))
    assert np.all(rest > 0)
    last = rng.standard_normal((n, d - m * k))
    last *= (np.sqrt(rest) / np.linalg.norm(last, axis=1))[:, None]
    y = np.concatenate([mid.reshape(n, m * k), last], axis=1)
    nu = np.exp(rng.uniform(-3.0, 3.0, size=(n, 1)))
    x = (nu * (y @ R.astype(np.float64))).astype(np.float32)
    xs = torch.from_numpy(x).to(dtype)
    _, _, D = occ.encode(gh.host_f64(xs), R.astype(np.float64), C64, return_distances=True)
    Dsort = np.sort(D, axis=-1)
    close = int(((Dsort[..., 1] - Dsort[..., 0]) <= 1e-3 * Dsort[..., 1]).sum())
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    _say(f"[edge] k={k} N={N} {dtype} near midpoints: {close} blocks within 1e-3 relative")
    assert close > 1000
    p, nrm = fq.encode(xs.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(xs), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")


@pytest.mark.parametrize("k,N", [(4, 256), (4, 64), (4, 16), (2, 64)])
def test_encode_k4_k2_many_out_of_range_rows(k, N, device):
    """bf16 rows at d = 64, k = 4 or 2, whose squared sums leave the float32
    range (every block of such a row is redone in float64): a 32-row tile
    with 16 of them (more blocks than the encoder's per-wavefront queue of
    deferred blocks holds), a lone one (k = 4: exactly a full queue), pairs
    and scattered rows up to the ragged last tile, among ordinary rows with
    their own near ties; every index must be the float64 argmin."""
    d = 64
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(41 + 7 * k + N)
    n = 1000
    x = torch.randn(n, d, generator=g) * torch.exp(torch.randn(n, 1, generator=g))
    for r in list(range(32, 48)) + [64, 130, 131, 200, 333, 517, 998, 999]:
        x[r] = (1e30 if r % 2 else 1e-30) * torch.randn(d, generator=g)
    x = x.to(torch.bfloat16)
    _say(f"[edge] bf16 k={k} N={N} many out-of-range rows")
    p, nrm = fq.encode(x.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(x), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_encode_k2_n64_grid_edge_cases(dtype, device):
    """k = 2, N = 64 at d = 64 (nearest codewords from a grid of the block
    plane): a cluster of ten codewords inside one grid cell (more candidates
    than a cell holds), a duplicated codeword (exact ties), blocks of y
    outside the grid's square (|y_b| up to 0.95), blocks at the cluster and at
    midpoints of neighbouring codewords, and ordinary rows; every index must
    be the float64 argmin (1e-6 window)."""
    d, k, N = 64, 2, 64
    R = oracle_rotation(d).astype(np.float64)
    C = quick_codebook(d, k, N).astype(np.float64)
    rng = np.random.default_rng(77)
    C[40:50] = np.array([0.101, 0.093]) + 0.004 * rng.standard_normal((10, 2))
    C[63] = C[5]
    C = C.astype(np.float32)
    C64 = C.astype(np.float64)
    D2 = ((C64[:, None, :] - C64[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(D2, np.inf)
    nbr = D2.argmin(1)
    n, nb = 6000, d // k
    y = rng.standard_normal((n, d))
    y /= np.linalg.norm(y, axis=1, keepdims=True)
    yb = y.reshape(n, nb, k)
    # rows 0 .. 999: blocks 0 .. 9 at the cluster; 1000 .. 1999: blocks
    # 0 .. 4 at midpoints; 2000 .. 2299: block 3 far out (|y_3| = 0.95); the
    # other blocks of these rows rescaled so that |y| = 1
    yb[:1000, :10] = np.array([0.101, 0.093]) + 0.01 * rng.standard_normal((1000, 10, 2))
    a = rng.integers(0, N, size=(1000, 5))
    yb[1000:2000, :5] = 0.5 * (C64[a] + C64[nbr[a]])
    ang = rng.uniform(0, 2 * np.pi, 300)
    yb[2000:2300, 3] = 0.95 * np.stack([np.cos(ang), np.sin(ang)], -1)
    y = yb.reshape(n, d)
    for lo, hi, keep in ((0, 1000, 10), (1000, 2000, 5), (2000, 2300, None)):
        rows = y[lo:hi]
        if keep is None:
            fixed = np.zeros(d, bool)
            fixed[6:8] = True
        else:
            fixed = np.zeros(d, bool)
            fixed[:2 * keep] = True
        rest = 1.0 - (rows[:, fixed] ** 2).sum(1)
        assert np.all(rest > 0)
        free = rows[:, ~fixed]
        rows[:, ~fixed] = free * (np.sqrt(rest) / np.linalg.norm(free, axis=1))[:, None]
    nu = np.exp(rng.uniform(-3.0, 3.0, size=(n, 1)))
    x = (nu * (y @ R)).astype(np.float32)
    xs = torch.from_numpy(x).to(dtype)
    Rd, Cd = torch.from_numpy(R.astype(np.float32)).to(device), torch.from_numpy(C.copy()).to(device)
    _say(f"[edge] k=2 N=64 {dtype} grid edge cases")
    p, nrm = fq.encode(xs.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(xs), R.astype(np.float32), C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")


@pytest.mark.parametrize("d,dtype,N,variant", [
    (128, torch.bfloat16, 4096, "fp16"), (128, torch.bfloat16, 4096, "plain"),
    (128, torch.float16, 2048, "dup"), (128, torch.float32, 1024, "plain"),
    (128, torch.bfloat16, 4096, "wide"),
    (64, torch.bfloat16, 256, "plain"), (64, torch.float16, 256, "dup"),
    (64, torch.float32, 1024, "fp16"), (64, torch.bfloat16, 4096, "wide"),
    (64, torch.bfloat16, 512, "plain")])
def test_encode_large_codebook_path(d, dtype, N, variant, device):
    """k = 4 with d = 128, N >= 1024 or d = 64, N in {256, 1024, 4096} (the
    matrix-core screen with its float64 certificate and full float64
    re-score; d = 64, N = 512 takes the general encoder): norms over several
    decades, zero rows, strided rows, a ragged count, codebooks with and
    without exact binary16 entries, duplicated codewords (exact ties: lowest
    index), and a codebook outside the screen's range (|c| > 2: every block
    re-scored)."""
    k = 4
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N).copy()
    if variant == "fp16":
        C = C.astype(np.float16).astype(np.float32)
    elif variant == "dup":  # the same codeword in two tiles, and twice in one tile
        C[N - 5] = C[40]
        C[9] = C[8]
    elif variant == "wide":
        C[17] *= 2.5 / np.linalg.norm(C[17])
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(N + len(variant))
    n = 333 if variant == "wide" else 1037
    x = torch.randn(n, 2 * d, generator=g) * torch.exp(2 * torch.randn(n, 1, generator=g))
    x[3] = 0
    x[20, :d] = 0
    x[20, d // 2 + 13] = 2.0 ** -20
    x = x.to(dtype)
    xs = x[:, :d]
    xd = x.to(device)[:, :d]
    assert xd.stride(0) == 2 * d
    _say(f"[edge] large codebook path d={d} dtype={dtype} N={N} variant={variant}")
    p, nrm = fq.encode(xd, k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(xs), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")
    assert not p.cpu().numpy()[3].any() and int(gh.bits_u16(nrm)[3]) == 0
    p2, n2 = fq.encode(xd.contiguous(), k, N, Rd, Cd)
    assert torch.equal(p, p2) and torch.equal(nrm, n2)


@pytest.mark.parametrize("k,N", [(8, 16), (4, 256)])
def test_decode_out_of_range_ids_give_nan(k, N, device):
    """Both decoders (the LDS table for small codebooks, the Pi^T product
    otherwise) return NaN rows for ids outside the cache."""
    d = 64
    R, C = oracle_rotation(d), quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    P = fq.payload_bytes(d, k, N)
    pay = torch.randint(0, 256, (100, P), dtype=torch.uint8).to(device)
    nb = torch.full((100,), 0x3C00, dtype=torch.int16).to(device)
    ids = torch.tensor([0, 99, 100, -1, 5], dtype=torch.int64).to(device)
    _say("[edge] decode ids out of range")
    out = fq.decode(pay, nb, d, k, N, Rd, Cd, token_ids=ids).cpu()
    assert torch.isnan(out[2]).all() and torch.isnan(out[3]).all()
    assert torch.isfinite(out[[0, 1, 4]]).all()


@pytest.mark.parametrize("T,T_stride,N,fp16_cb", [(0, 16, 64, False), (1, 8, 64, False),
                                                   (65, 80, 64, False), (1000, 1100, 64, False),
                                                   (70, 73, 16, False), (700, 701, 16, True),
                                                   (2047, 2048, 64, True), (33, 33, 16, True)])
def test_attention_token_counts(T, T_stride, N, fp16_cb, device):
    """T = 0 writes zeros; T = 1 returns the single value; ragged tails and
    T_stride > T (bytes beyond T are junk and must be ignored)."""
    d, k, G = 64, 8, 8
    R, C = oracle_rotation(d), quick_codebook(d, k, N)
    if fp16_cb:  # a codebook whose entries are exactly representable in binary16
        C = C.astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    n_g = 3
    rng = np.random.default_rng(T)
    P = occ.payload_bytes(d, k, N)
    idx_k = rng.integers(0, N, (n_g, T_stride, d // k))
    idx_v = rng.integers(0, N, (n_g, T_stride, d // k))
    hk = (np.abs(rng.standard_normal((n_g, T_stride))) * 30).astype(np.float16)
    hv = (np.abs(rng.standard_normal((n_g, T_stride))) * 30).astype(np.float16)
    kp = occ.pack(idx_k.reshape(-1, d // k), N).reshape(n_g, T_stride, P)
    vp = occ.pack(idx_v.reshape(-1, d // k), N).reshape(n_g, T_stride, P)
    q = rng.standard_normal((n_g, G, d)).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    _say(f"[edge] attention T={T} T_stride={T_stride} N={N} fp16 codebook={fp16_cb}")
    o = fq.attn_decode(dev(q), dev(kp), dev(occ.fp16_bits(hk).view(np.int16)), dev(vp),
                       dev(occ.fp16_bits(hv).view(np.int16)), T, k, N, Rd, Cd).cpu().numpy()
    if T == 0:
        assert np.all(o == 0)
        return
    ref = gh.oracle_group_attention(q.astype(np.float64), kp, occ.fp16_bits(hk), vp,
                                    occ.fp16_bits(hv), R, C, N, T)
    gh.check_attention(o, ref)


def _random_attention_inputs(rng, n_g, T, d, k, N, G, kscale=30.0):
    P = occ.payload_bytes(d, k, N)
    idx_k = rng.integers(0, N, (n_g * T, d // k))
    idx_v = rng.integers(0, N, (n_g * T, d // k))
    hk = (np.abs(rng.standard_normal(n_g * T)) * kscale).astype(np.float16).reshape(n_g, T)
    hv = (np.abs(rng.standard_normal(n_g * T)) * 30).astype(np.float16).reshape(n_g, T)
    kp = occ.pack(idx_k, N).reshape(n_g, T, P)
    vp = occ.pack(idx_v, N).reshape(n_g, T, P)
    q = rng.standard_normal((n_g, G, d)).astype(np.float32)
    return q, kp, hk, vp, hv


@pytest.mark.parametrize("N,n_g,T", [(16, 1100, 70), (16, 600, 300), (64, 1100, 70)])
def test_attention_many_short_groups(N, n_g, T, device):
    """Many short groups: each workgroup of the sub-one-bit kernels meets
    more groups than it keeps query operands for, which takes the 4-bit
    kernel's three-launch form (a separate query preparation kernel)."""
    d, k, G = 64, 8, 8
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N).astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    rng = np.random.default_rng(n_g + T)
    q, kp, hk, vp, hv = _random_attention_inputs(rng, n_g, T, d, k, N, G)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    _say(f"[edge] attention many short groups N={N} n_g={n_g} T={T}")
    o = fq.attn_decode(dev(q), dev(kp), dev(occ.fp16_bits(hk).view(np.int16)), dev(vp),
                       dev(occ.fp16_bits(hv).view(np.int16)), T, k, N, Rd, Cd).cpu().numpy()
    ref = gh.oracle_group_attention(q.astype(np.float64), kp, occ.fp16_bits(hk), vp,
                                    occ.fp16_bits(hv), R, C, N, T)
    gh.check_attention(o, ref)


def test_attention_workspace_reuse_across_shapes(device):
    """One workspace serves a sequence of calls of different shapes and
    kernels (the two-launch and three-launch forms of the 4-bit kernel, the
    6-bit kernel, the k = 4 kernel): whatever an earlier call left in it,
    every result matches the oracle."""
    d, G = 64, 8
    R = oracle_rotation(d)
    Rd = torch.from_numpy(R.copy()).to(device)
    calls = [(8, 16, 5, 5000), (8, 16, 1100, 70), (8, 64, 4, 3000), (4, 256, 6, 700),
             (8, 16, 3, 7777), (8, 16, 5, 5000)]
    books = {}
    need = max(fq.attn_workspace_bytes(n_g, G, T, d, k, N) for k, N, n_g, T in calls)
    ws = torch.full((need,), 0xA5, dtype=torch.uint8, device=device)  # junk, not zeros
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    for i, (k, N, n_g, T) in enumerate(calls):
        if (k, N) not in books:
            books[(k, N)] = quick_codebook(d, k, N).astype(np.float16).astype(np.float32)
        C = books[(k, N)]
        rng = np.random.default_rng(100 + i)
        q, kp, hk, vp, hv = _random_attention_inputs(rng, n_g, T, d, k, N, G)
        _say(f"[edge] workspace reuse call {i}: k={k} N={N} n_g={n_g} T={T}")
        o = fq.attn_decode(dev(q), dev(kp), dev(occ.fp16_bits(hk).view(np.int16)), dev(vp),
                           dev(occ.fp16_bits(hv).view(np.int16)), T, k, N, Rd,
                           torch.from_numpy(C.copy()).to(device), workspace=ws).cpu().numpy()
        ref = gh.oracle_group_attention(q.astype(np.float64), kp, occ.fp16_bits(hk), vp,
                                        occ.fp16_bits(hv), R, C, N, T)
        gh.check_attention(o, ref)


@pytest.mark.parametrize("N", [16, 64])
def test_attention_huge_query_small_keys(N, device):
    """Rotated query entries far beyond binary16 range (the matrix-core path
    rescales them by a power of two) against tiny key norms, so the logits
    stay moderate and the softmax is well conditioned."""
    d, k, G, T, n_g = 64, 8, 8, 700, 3
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N).astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    rng = np.random.default_rng(11)
    P = occ.payload_bytes(d, k, N)
    idx_k = rng.integers(0, N, (n_g * T, d // k))
    idx_v = rng.integers(0, N, (n_g * T, d // k))
    hk = (np.abs(rng.standard_normal(n_g * T)) * 2e-4 + 1e-4).astype(np.float16)
    hv = (np.abs(rng.standard_normal(n_g * T)) * 10).astype(np.float16)
    kp = occ.pack(idx_k, N).reshape(n_g, T, P)
    vp = occ.pack(idx_v, N).reshape(n_g, T, P)
    q = (rng.standard_normal((n_g, G, d)) * 3e5).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    _say(f"[edge] attention huge query N={N}")
    o = fq.attn_decode(dev(q), dev(kp), dev(occ.fp16_bits(hk).view(np.int16).reshape(n_g, T)),
                       dev(vp), dev(occ.fp16_bits(hv).view(np.int16).reshape(n_g, T)), T, k, N,
                       Rd, Cd).cpu().numpy()
    ref = gh.oracle_group_attention(q.astype(np.float64), kp, occ.fp16_bits(hk).reshape(n_g, T), vp,
                                    occ.fp16_bits(hv).reshape(n_g, T), R, C, N, T)
    gh.check_attention(o, ref)


@pytest.mark.parametrize("d,k,N,G,T,T_stride,fp16_cb,qmul", [
    (64, 4, 256, 8, 700, 733, False, 1.0), (64, 4, 256, 1, 33, 33, True, 1.0),
    (64, 4, 256, 5, 1, 8, False, 1.0), (128, 4, 4096, 4, 1000, 1029, True, 1.0),
    (128, 4, 4096, 4, 65, 65, False, 3e5), (128, 4, 256, 8, 517, 600, True, 1.0),
    (64, 4, 256, 8, 0, 16, False, 1.0), (64, 4, 4096, 8, 300, 301, False, 1.0),
    (64, 2, 64, 8, 700, 733, False, 1.0), (64, 2, 16, 1, 33, 33, True, 1.0),
    (64, 2, 64, 4, 65, 65, False, 3e5), (128, 2, 64, 4, 1000, 1029, True, 1.0),
    (128, 2, 16, 8, 517, 600, False, 1.0), (64, 2, 64, 8, 0, 16, False, 1.0)])
def test_attention_k4_shapes(d, k, N, G, T, T_stride, fp16_cb, qmul, device):
    """Block dimension k = 4 (the matrix-core path for 8- and 12-bit
    indices) and k = 2 with 4- or 6-bit indices (read by the same path as
    pairs of blocks over the pair codebook): ragged T, T_stride > T, G below
    8, a single token, T = 0, codebooks with and without exact binary16
    entries, and rotated queries far beyond binary16 range against small key
    norms."""
    R, C = oracle_rotation(d), quick_codebook(d, k, N)
    if fp16_cb:
        C = C.astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    n_g = 3
    rng = np.random.default_rng(T + d + G)
    P = occ.payload_bytes(d, k, N)
    idx_k = rng.integers(0, N, (n_g, T_stride, d // k))
    idx_v = rng.integers(0, N, (n_g, T_stride, d // k))
    kscale = 30.0 / qmul if qmul > 1 else 30.0
    hk = (np.abs(rng.standard_normal((n_g, T_stride))) * kscale).astype(np.float16)
    hv = (np.abs(rng.standard_normal((n_g, T_stride))) * 30).astype(np.float16)
    kp = occ.pack(idx_k.reshape(-1, d // k), N).reshape(n_g, T_stride, P)
    vp = occ.pack(idx_v.reshape(-1, d // k), N).reshape(n_g, T_stride, P)
    q = (rng.standard_normal((n_g, G, d)) * qmul).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    _say(f"[edge] attention k={k} d={d} N={N} G={G} T={T} T_stride={T_stride} fp16={fp16_cb} q x{qmul:g}")
    o = fq.attn_decode(dev(q), dev(kp), dev(occ.fp16_bits(hk).view(np.int16)), dev(vp),
                       dev(occ.fp16_bits(hv).view(np.int16)), T, k, N, Rd, Cd).cpu().numpy()
    if T == 0:
        assert np.all(o == 0)
        return
    ref = gh.oracle_group_attention(q.astype(np.float64), kp, occ.fp16_bits(hk), vp,
                                    occ.fp16_bits(hv), R, C, N, T)
    gh.check_attention(o, ref)


def test_attention_zero_query_is_mean_value(device):
    """q = 0: every score is 0, the output is the mean decoded value."""
    d, k, N, G, T = 128, 4, 4096, 4, 300
    R, C = oracle_rotation(d), quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    rng = np.random.default_rng(3)
    idx = rng.integers(0, N, (T, d // k))
    h = (np.abs(rng.standard_normal(T)) * 10).astype(np.float16)
    pay = occ.pack(idx, N)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    nb = occ.fp16_bits(h).view(np.int16)
    _say("[edge] attention zero query")
    o = fq.attn_decode(dev(np.zeros((1, G, d), np.float32)), dev(pay[None]), dev(nb[None]),
                       dev(pay[None]), dev(nb[None]), T, k, N, Rd, Cd).cpu().numpy()
    mean = occ.decode(idx, h, R.astype(np.float64), C.astype(np.float64)).mean(0)
    gh.check_attention(o[0], np.repeat(mean[None], G, 0))


@pytest.mark.parametrize("d,k,N", [(64, 1, 4), (64, 1, 8), (64, 1, 16), (128, 1, 16), (64, 2, 128),
                                   (64, 2, 256), (64, 16, 8192), (64, 4, 1024), (128, 4, 1024),
                                   (64, 8, 256), (64, 8, 1024), (64, 16, 256), (64, 16, 1024),
                                   (64, 8, 4096), (128, 8, 4096), (64, 16, 4096),
                                   (64, 32, 1024), (64, 32, 16384), (64, 64, 1024), (64, 64, 16384)])
def test_rate_axis_operating_points(d, k, N, device):
    """Operating points of the paper's rate axis beyond the benchmark
    workloads (the scalar k = 1 code, k = 4 at N = 1024 with 10-bit indices in
    a 20-byte payload (the Sec. 5.3 TinyLlama table's k = 4, N = 1024 row),
    larger codebooks at k = 2, 8, 16, up to
    the 128 and 256 KB codebooks of k = 8 and 16 at N = 4096, read from
    global memory) and the large-block codes k = 32, 64 (k = d: one codeword
    per vector, N up to 16384, a 4 MB codebook) through the general kernels:
    encode, range and random-access decode and fused attention against the
    oracle on a bf16 cache with heavy-tailed channel scales (2 groups x 333
    tokens, G = 4).  Codec parity holds for any codebook: the large-block
    points and codebooks above 256 KB use seeded random codewords (norms in
    [0.4, 1]) instead of a Lloyd build."""
    R = oracle_rotation(d)
    if k >= 32 or N * k > 65536:  # an oracle Lloyd build would take minutes
        rng = np.random.default_rng(7 + k + N)
        C = rng.standard_normal((N, k))
        C *= rng.uniform(0.4, 1.0, (N, 1)) / np.linalg.norm(C, axis=1, keepdims=True)
        C = C.astype(np.float32)
    else:
        C = quick_codebook(d, k, N)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    n_g, T, G = 2, 333, 4
    g = torch.Generator().manual_seed(1000 * k + N + d)
    sig = torch.exp(0.5 * torch.randn(1, d, generator=g))
    sig[0, :2] *= 10
    kx = (torch.randn(n_g * T, d, generator=g) * sig).to(torch.bfloat16)
    vx = (torch.randn(n_g * T, d, generator=g) * sig).to(torch.bfloat16)
    q = torch.randn(n_g, G, d, generator=g).to(torch.bfloat16)
    _say(f"[rate axis] d={d} k={k} N={N}")
    kp, kn = fq.encode(kx.to(device), k, N, Rd, Cd)
    vp, vn = fq.encode(vx.to(device), k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, k_idx, k_h = gh.check_encode(gh.host_f64(kx), R, C, N, kp, kn)
    ne2, nt2, v_idx, v_h = gh.check_encode(gh.host_f64(vx), R, C, N, vp, vn)
    _say(f"  encode: {ne + ne2} exact indices, {nt + nt2} accepted near-ties")
    k_pay, v_pay = occ.pack(k_idx, N), occ.pack(v_idx, N)
    k_nb, v_nb = occ.fp16_bits(k_h), occ.fp16_bits(v_h)
    pd = torch.from_numpy(k_pay).to(device)
    nd = torch.from_numpy(k_nb.view(np.int16)).to(device)
    xh = fq.decode(pd, nd, d, k, N, Rd, Cd)
    gh.check_recon(xh.cpu().numpy(), occ.decode(k_idx, k_h, R.astype(np.float64), C.astype(np.float64)), k_h)
    ids = torch.tensor([0, 5, n_g * T - 1, 77], dtype=torch.int64)
    xs = fq.decode(pd, nd, d, k, N, Rd, Cd, token_ids=ids.to(device))
    assert torch.equal(xs.cpu(), xh.cpu()[ids])
    P = k_pay.shape[1]
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    o = fq.attn_decode(q.to(device), t(k_pay.reshape(n_g, T, P)), t(k_nb.view(np.int16).reshape(n_g, T)),
                       t(v_pay.reshape(n_g, T, P)), t(v_nb.view(np.int16).reshape(n_g, T)), T, k, N,
                       Rd, Cd)
    ref = gh.oracle_group_attention(gh.host_f64(q), k_pay.reshape(n_g, T, P), k_nb.reshape(n_g, T),
                                    v_pay.reshape(n_g, T, P), v_nb.reshape(n_g, T), R, C, N, T)
    rel = gh.check_attention(o.cpu().numpy(), ref)
    _say(f"  attention: max rel l2 {rel:.2e}")


def _check_radius_first(x64, R, C, L, payload, norms, k, N):
    """Headers bit-exact; indices equal to the oracle's radius-first search, or
    (floating-point ties only) a shell no farther in radius by 1e-12 and,
    inside it, a codeword within the 1e-6 distance window."""
    d = R.shape[0]
    idx_ref, h_ref, shell_ref = osl.encode_radius_first(x64, R, C, L)
    idx_gpu = occ.unpack(payload.cpu().numpy(), d // k, N)
    assert np.array_equal(gh.bits_u16(norms), occ.fp16_bits(h_ref))
    bad = idx_gpu != idx_ref
    if bad.any():
        nu, _ = occ.norms(x64)
        y = occ.rotate_normalise(x64, R.astype(np.float64), nu).reshape(x64.shape[0], d // k, k)
        r = osl.shell_radii(d, k, L)
        Ma = N // L
        for v, m in zip(*np.nonzero(bad)):
            b = y[v, m]
            rho = float(np.linalg.norm(b))
            lg = int(idx_gpu[v, m]) // Ma
            assert abs(rho - r[lg]) <= abs(rho - r[shell_ref[v, m]]) + 1e-12, (v, m)
            D = ((b[None, :] - C[lg * Ma:(lg + 1) * Ma].astype(np.float64)) ** 2).sum(1)
            assert D[idx_gpu[v, m] - lg * Ma] <= D.min() * (1 + gh.TIE_REL), (v, m)
    return int((~bad).sum()), int(bad.sum())


@pytest.mark.parametrize("d,k,N,L,dtype", [
    (64, 4, 256, 16, torch.bfloat16), (64, 8, 1024, 32, torch.float16),
    (128, 4, 4096, 64, torch.bfloat16), (64, 2, 64, 8, torch.float32),
    (64, 4, 256, 1, torch.bfloat16), (64, 16, 4096, 64, torch.float32),
    (64, 32, 8192, 128, torch.bfloat16), (128, 8, 256, 256, torch.float16)])
def test_encode_radius_first_parity(d, k, N, L, dtype, device):
    """fibq_encode_radius_first (App. F Stage 1) against the oracle's
    radius-first search on a multi-shell codebook C(L, N/L) whose codewords
    are moved off their shells (as a Lloyd polish does): strided rows, a
    ragged count, a zero row and norms over several decades; codebooks above
    64 KB are read from global memory; L = 1 is the exhaustive search and
    M_a = 1 (L = N) a pure radius choice."""
    rng = np.random.default_rng(N + L + k)
    C0 = ocb.multishell_codebook(d, k, L, N // L)
    C = (C0 * (1 + 0.05 * rng.standard_normal((N, 1)))
         + 0.01 * rng.standard_normal((N, k)) * np.linalg.norm(C0, axis=1, keepdims=True))
    C = C.astype(np.float32)
    R = oracle_rotation(d)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(N + L)
    n = 1037
    x = torch.randn(n, 2 * d, generator=g) * torch.exp(2 * torch.randn(n, 1, generator=g))
    x[3] = 0
    x = x.to(dtype)
    xd = x.to(device)[:, :d]
    _say(f"[radius-first] d={d} k={k} N={N} L={L} dtype={dtype}")
    p, nrm = fq.encode_radius_first(xd, k, N, L, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt = _check_radius_first(gh.host_f64(x[:, :d]), R, C, L, p, nrm, k, N)
    _say(f"  {ne} exact indices, {nt} accepted floating-point ties")
    assert not p.cpu().numpy()[3].any() and int(gh.bits_u16(nrm)[3]) == 0


def test_encode_radius_first_rejects_bad_shell_counts(device):
    R = torch.from_numpy(oracle_rotation(64).copy()).to(device)
    C = torch.zeros((256, 4), device=device)
    x = torch.zeros((8, 64), device=device)
    for L in (0, 3, 512):
        with pytest.raises(fq.FibqError) as e:
            fq.encode_radius_first(x, 4, 256, L, R, C)
        assert e.value.status == fq.FIBQ_EINVAL


@pytest.mark.parametrize("d,k,N,L,K,T,dtype", [
    (64, 4, 256, 16, 4, 1, torch.bfloat16), (64, 4, 256, 16, 4, 2, torch.float16),
    (64, 8, 1024, 32, 4, 4, torch.float32), (128, 4, 4096, 64, 8, 2, torch.bfloat16),
    (64, 32, 8192, 64, 8, 3, torch.bfloat16)])
def test_encode_list_parity(d, k, N, L, K, T, dtype, device):
    """fibq_encode_list (App. F Stages 1 + 2) against the oracle's list
    decoding with the same parent tables (the oracle's): equal indices, or
    (floating-point ties only) a candidate no farther than the oracle's by
    1e-6 relative, from the same shell up to a 1e-12 radius tie and from a
    parent within 1e-9 of the T-th best score.  T = K is the radius-first
    search."""
    rng = np.random.default_rng(N + L + K + T)
    C0 = ocb.multishell_codebook(d, k, L, N // L)
    C = (C0 * (1 + 0.05 * rng.standard_normal((N, 1)))
         + 0.01 * rng.standard_normal((N, k)) * np.linalg.norm(C0, axis=1, keepdims=True))
    C = C.astype(np.float32)
    mu, groups = osl.parent_tables(C.astype(np.float64), L, K)
    Ma = N // L
    off = np.zeros((L, K + 1), dtype=np.int32)
    mem = np.zeros(N, dtype=np.int32)
    for l in range(L):
        pos = 0
        for p in range(K):
            off[l, p] = pos
            ids = np.flatnonzero(groups[l * Ma:(l + 1) * Ma] == p)
            mem[l * Ma + pos:l * Ma + pos + ids.size] = ids
            pos += ids.size
        off[l, K] = pos
    R = oracle_rotation(d)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    mud = torch.from_numpy(mu.copy()).to(device)
    offd = torch.from_numpy(off).to(device)
    memd = torch.from_numpy(mem).to(device)
    g = torch.Generator().manual_seed(N + K + T)
    n = 777
    x = torch.randn(n, 2 * d, generator=g) * torch.exp(2 * torch.randn(n, 1, generator=g))
    x[5] = 0
    x = x.to(dtype)
    xd = x.to(device)[:, :d]
    _say(f"[list] d={d} k={k} N={N} L={L} K={K} T={T} dtype={dtype}")
    p, nrm = fq.encode_list(xd, k, N, L, K, T, mud, offd, memd, Rd, Cd)
    torch.cuda.synchronize()
    x64 = gh.host_f64(x[:, :d])
    idx_ref, h_ref = osl.encode_hierarchical_tables(x64, R.astype(np.float64), C.astype(np.float64),
                                                    L, mu, groups, T)
    idx_gpu = occ.unpack(p.cpu().numpy(), d // k, N)
    assert np.array_equal(gh.bits_u16(nrm), occ.fp16_bits(h_ref))
    bad = np.argwhere(idx_gpu != idx_ref)
    if bad.size:
        nu, _ = occ.norms(x64)
        y = occ.rotate_normalise(x64, R.astype(np.float64), nu).reshape(n, d // k, k)
        r = osl.shell_radii(d, k, L)
        C64 = C.astype(np.float64)
        for v, m in bad:
            b = y[v, m]
            rho = float(np.linalg.norm(b))
            jg, jo = int(idx_gpu[v, m]), int(idx_ref[v, m])
            lg, lo = jg // Ma, jo // Ma
            assert abs(rho - r[lg]) <= abs(rho - r[lo]) + 1e-12, (v, m)
            sc = mu[lg] @ b
            assert sc[groups[jg]] >= np.sort(sc)[::-1][T - 1] - 1e-9, (v, m)
            dg, do = ((b - C64[jg]) ** 2).sum(), ((b - C64[jo]) ** 2).sum()
            assert dg <= do * (1 + gh.TIE_REL), (v, m)
    _say(f"  {idx_gpu.size - len(bad)} exact indices, {len(bad)} accepted floating-point ties")
    assert not p.cpu().numpy()[5].any()
    if T == K:
        p2, _ = fq.encode_radius_first(xd, k, N, L, Rd, Cd)
        assert torch.equal(p, p2)


@pytest.mark.parametrize("k,N,dtype", [(32, 2048, torch.bfloat16), (64, 1024, torch.float16)])
def test_encode_chunked_large_blocks_edge_cases(k, N, dtype, device):
    """The large-block encoder that stages the codebook through LDS (d = 64,
    k >= 32, codebooks above 64 KB): strided rows, a zero row, a tiny-norm
    row and a ragged count across several 256-vector tiles."""
    d = 64
    R = oracle_rotation(d)
    rng = np.random.default_rng(k + N)
    C = rng.standard_normal((N, k))
    C = (C * rng.uniform(0.4, 1.0, (N, 1)) / np.linalg.norm(C, axis=1, keepdims=True)).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    g = torch.Generator().manual_seed(k + N)
    n = 601
    x = torch.randn(n, 2 * d, generator=g) * torch.exp(2 * torch.randn(n, 1, generator=g))
    x[7] = 0
    x[300, :d] = 0
    x[300, 5] = 2.0 ** -20
    x = x.to(dtype)
    xd = x.to(device)[:, :d]
    _say(f"[edge] chunked large-block encoder k={k} N={N} dtype={dtype}")
    p, nrm = fq.encode(xd, k, N, Rd, Cd)
    torch.cuda.synchronize()
    ne, nt, _, _ = gh.check_encode(gh.host_f64(x[:, :d]), R, C, N, p, nrm)
    _say(f"  {ne} exact indices, {nt} accepted near-ties")
    assert not p.cpu().numpy()[7].any() and int(gh.bits_u16(nrm)[7]) == 0
