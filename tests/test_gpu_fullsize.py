"""Parity at full workload sizes, in the launch configuration the benchmark
times: one encode call per cache and one attention call over all groups
(many token units per wavefront, groups shared between workgroups).  The
float64 oracle cannot encode whole caches of tens of millions of vectors, so
it checks sampled outputs it computes one by one:

  * encode: seeded random rows plus the first and last 64 rows of each cache
    (indices up to the near-tie rule, payload bytes and header bits);
  * attention: whole groups (the first two, a middle one, the last, and for
    the 4-bit kernel groups its plan splits between workgroups).  Where the
    oracle can encode a group in seconds it does, and its payload is written
    into the device buffers in place of the device's own; for the
    4096-codeword workload the device's own payload of those groups (already
    checked row by row above) is the input.  The full call runs, and those
    groups' outputs are compared with naive oracle attention on the same
    payload.

Workloads: the 32k-context cache (22 x 4 x 4 groups x 32768 tokens, both
rates), the TinyLlama-shaped cache (22 x 8 x 4 groups x 2048 tokens, both
rates), the GPT-2-shaped cache (144 groups x 1024 tokens) and the stress cache
(32 x 8 groups x 131072 tokens, d = 128, N = 4096).
"""
import numpy as np
import pytest
import torch

import paper_2605_11478_amd as fq
from paper_2605_11478_amd import workloads as W
from oracle import codec as occ

from _fixtures import oracle_rotation, quick_codebook
import gpu_helpers as gh

pytestmark = pytest.mark.gpu

FULL = [("long32k", 0), ("long32k", 1), ("tinyllama", 0), ("tinyllama", 1), ("gpt2", 0),
        ("stress", 0)]
ORACLE_GROUP_WORK = 2 ** 27  # T x (d / k) x N above which the oracle does not encode groups


def _say(*a):
    print(*a, flush=True)


def w4_split_groups(n_g, T, unit=128, max_wgs=256):
    """Groups whose tokens the 4-bit fused attention (d = 64, k = 8, N = 16,
    G = 8) splits between two or more workgroups: the cache of all groups is
    laid end to end as `unit`-token units and workgroup w of min(units,
    max_wgs) owns units [w units / wgs, (w + 1) units / wgs)."""
    upg = -(-T // unit)
    units = n_g * upg
    wgs = min(units, max_wgs)
    starts = [(w * units) // wgs for w in range(wgs)]
    owner = lambda u: max(w for w in range(wgs) if starts[w] <= u)
    return [g for g in range(n_g) if owner(g * upg) != owner((g + 1) * upg - 1)]


def sample_groups(name, rate, n_g, T):
    """The first, second, a middle and the last group; for the 4-bit fused
    attention also the first groups its plan splits between workgroups (their
    records are merged across workgroups), checked to be among them."""
    groups = sorted({0, 1, n_g // 2 + 3, n_g - 1})
    wl = W.WORKLOADS[name]
    if (wl.d, *wl.rates[rate], wl.G) == (64, 8, 16, 8):
        split = w4_split_groups(n_g, T)
        assert split, "the plan splits no group"
        groups = sorted(set(groups) | set(split[:2]))
        assert set(groups) & set(split)
    return groups


@pytest.mark.parametrize("name,rate", FULL)
def test_full_size_sampled(name, rate, device):
    wl = W.WORKLOADS[name]
    k, N = wl.rates[rate]
    d, G, T, n_g = wl.d, wl.G, wl.T, wl.n_groups
    # the oracle's codebook, rounded to binary16 as the library's builder does
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N).astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    _say(f"[full size] {name} k={k} N={N}: {2 * n_g * T} vectors")
    kc = W.make_cache(wl, "k", device)
    vc = W.make_cache(wl, "v", device)
    q = W.group_view_query(W.make_query(wl, device), wl)
    kx, vx = kc.reshape(-1, d), vc.reshape(-1, d)
    n_v = kx.shape[0]
    kp, kn = fq.encode(kx, k, N, Rd, Cd)
    vp, vn = fq.encode(vx, k, N, Rd, Cd)
    torch.cuda.synchronize()

    rng = np.random.default_rng(100 + rate + 10 * len(name))
    n_rand = 3000 if N <= 256 else 600
    rows = np.unique(np.concatenate([rng.integers(0, n_v, n_rand), np.arange(64),
                                     np.arange(n_v - 64, n_v)]))
    ri = torch.from_numpy(rows).to(device)
    for tag, x, p, nrm in (("K", kx, kp, kn), ("V", vx, vp, vn)):
        ne, nt, _, _ = gh.check_encode(gh.host_f64(x[ri]), R, C, N, p[ri], nrm[ri])
        _say(f"  encode {tag}: {len(rows)} sampled rows, {ne} exact indices, {nt} near-ties")

    P = kp.shape[1]
    groups = sample_groups(name, rate, n_g, T)
    kpg, vpg = kp.view(n_g, T, P), vp.view(n_g, T, P)
    kng, vng = kn.view(n_g, T), vn.view(n_g, T)
    own = T * (d // k) * N > ORACLE_GROUP_WORK
    ref_pay = {}
    for g in groups:
        if own:  # the device's payload of this group
            ref_pay[g] = (kpg[g].cpu().numpy(), gh.bits_u16(kng[g]), vpg[g].cpu().numpy(),
                          gh.bits_u16(vng[g]))
            continue
        xk = gh.host_f64(kx[g * T:(g + 1) * T])
        xv = gh.host_f64(vx[g * T:(g + 1) * T])
        ik, hk, _ = gh.oracle_encode(xk, R, C)
        iv, hv, _ = gh.oracle_encode(xv, R, C)
        ref_pay[g] = (occ.pack(ik, N), occ.fp16_bits(hk), occ.pack(iv, N), occ.fp16_bits(hv))
        kpg[g].copy_(torch.from_numpy(ref_pay[g][0]))
        kng[g].copy_(torch.from_numpy(ref_pay[g][1].view(np.int16)))
        vpg[g].copy_(torch.from_numpy(ref_pay[g][2]))
        vng[g].copy_(torch.from_numpy(ref_pay[g][3].view(np.int16)))
    o = fq.attn_decode(q, kpg, kng, vpg, vng, T, k, N, Rd, Cd).cpu().numpy()
    qh = gh.host_f64(q)
    for g in groups:
        kpay, knb, vpay, vnb = ref_pay[g]
        ref = gh.oracle_group_attention(qh[g:g + 1], kpay[None], knb[None], vpay[None], vnb[None],
                                        R, C, N, T)
        rel = gh.check_attention(o[g:g + 1], ref)
        _say(f"  attention group {g}: max rel l2 {rel:.2e}")
    assert np.isfinite(o).all()


@pytest.mark.parametrize("name,L", [("gpt2", 16), ("tinyllama", 16), ("stress", 64)])
def test_full_size_radius_first_sampled(name, L, device):
    """The radius-first and list-decoding encoders (App. F) on the whole K
    cache, as `bench.py --radius-first` runs them, checked on sampled rows
    against the oracle's searches with the same multi-shell codebook and
    parent tables (indices up to floating-point ties, headers bit-exact)."""
    from oracle import codebook as ocb
    from oracle import sublinear as osl
    wl = W.WORKLOADS[name]
    k, N = wl.rates[0]
    d = wl.d
    Ma = N // L
    R = oracle_rotation(d)
    rng = np.random.default_rng(N + L)
    C0 = ocb.multishell_codebook(d, k, L, Ma)
    C = (C0 * (1 + 0.05 * rng.standard_normal((N, 1)))).astype(np.float32)
    Kp, T = (4, 2) if Ma <= 16 else (8, 2)
    mu, groups = osl.parent_tables(C.astype(np.float64), L, Kp)
    off = np.zeros((L, Kp + 1), dtype=np.int32)
    mem = np.zeros(N, dtype=np.int32)
    for l in range(L):
        pos = 0
        for p in range(Kp):
            off[l, p] = pos
            ids = np.flatnonzero(groups[l * Ma:(l + 1) * Ma] == p)
            mem[l * Ma + pos:l * Ma + pos + ids.size] = ids
            pos += ids.size
        off[l, Kp] = pos
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    kx = W.make_cache(wl, "k", device).reshape(-1, d)
    n_v = kx.shape[0]
    _say(f"[full size] radius-first {name} L={L}: {n_v} vectors")
    p1, n1 = fq.encode_radius_first(kx, k, N, L, Rd, Cd)
    p2, n2 = fq.encode_list(kx, k, N, L, Kp, T, torch.from_numpy(mu).to(device),
                            torch.from_numpy(off).to(device), torch.from_numpy(mem).to(device),
                            Rd, Cd)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(64), n_v - 64 + np.arange(64),
                                     np.random.default_rng(5).integers(0, n_v, 1500)]))
    rows_d = torch.from_numpy(rows).to(device)
    x64 = gh.host_f64(kx[rows_d])
    r = osl.shell_radii(d, k, L)
    nu, _ = occ.norms(x64)
    y = occ.rotate_normalise(x64, R.astype(np.float64), nu).reshape(len(rows), d // k, k)
    C64 = C.astype(np.float64)
    for label, pay, nrm, ref in (
            ("radius-first", p1, n1, osl.encode_radius_first(x64, R, C64, L)[:2]),
            ("list", p2, n2, osl.encode_hierarchical_tables(x64, R, C64, L, mu, groups, T))):
        idx_ref, h_ref = ref
        idx = occ.unpack(pay[rows_d].cpu().numpy(), d // k, N)
        assert np.array_equal(gh.bits_u16(nrm[rows_d]), occ.fp16_bits(h_ref)), label
        bad = np.argwhere(idx != idx_ref)
        for v, m in bad:  # floating-point ties only
            b = y[v, m]
            jg, jo = int(idx[v, m]), int(idx_ref[v, m])
            rho = float(np.linalg.norm(b))
            assert abs(rho - r[jg // Ma]) <= abs(rho - r[jo // Ma]) + 1e-12, (label, v, m)
            assert ((b - C64[jg]) ** 2).sum() <= ((b - C64[jo]) ** 2).sum() * (1 + gh.TIE_REL), \
                (label, v, m)
        _say(f"  {label}: {idx.size - len(bad)} exact indices, {len(bad)} accepted ties")


@pytest.mark.parametrize("k,N", [(16, 4096), (32, 16384), (64, 16384)])
def test_full_size_rate_axis_encode_sampled(k, N, device):
    """Rate-axis points on the whole GPT-2-shaped K cache, as `bench.py
    --rate-axis` encodes it: the general encoder with the row streamed from
    cache (k = 16) and the LDS-chunked large-block encoder (k = 32, 64),
    sampled rows against the oracle (indices up to the near-tie rule)."""
    wl = W.WORKLOADS["gpt2"]
    d = wl.d
    R = oracle_rotation(d)
    rng = np.random.default_rng(7 + k + N)
    C = rng.standard_normal((N, k))
    C = (C * rng.uniform(0.4, 1.0, (N, 1)) / np.linalg.norm(C, axis=1, keepdims=True)).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    kx = W.make_cache(wl, "k", device).reshape(-1, d)
    n_v = kx.shape[0]
    _say(f"[full size] rate axis k={k} N={N}: {n_v} vectors")
    p, nrm = fq.encode(kx, k, N, Rd, Cd)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(64), n_v - 64 + np.arange(64),
                                     np.random.default_rng(3).integers(0, n_v, 600)]))
    rows_d = torch.from_numpy(rows).to(device)
    ne, nt, _, _ = gh.check_encode(gh.host_f64(kx[rows_d]), R, C, N, p[rows_d], nrm[rows_d])
    _say(f"  {ne} exact indices, {nt} accepted near-ties")
