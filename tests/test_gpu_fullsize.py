"""Parity at the full 32k-context size (22 layers x 4 batch x 4 KV heads x
32768 tokens, d=64, bf16 K/V, G=8), in the launch configuration the benchmark
times: one encode call per cache and one attention call over all 352 groups.
The float64 oracle cannot encode 23 million vectors, so it checks sampled
outputs it computes one by one:

  * encode: ~3000 seeded random rows plus the first and last 64 rows of each
    cache (indices up to the near-tie rule, payload bytes and header bits);
  * attention: the oracle encodes three whole groups (first, a middle one,
    last) itself; that payload is written into the device buffers in place of
    the device's own, the full 352-group call runs, and those groups' outputs
    are compared with naive oracle attention on the oracle payload.
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


def _say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("rate", [0, 1])
def test_long32k_full_size_sampled(rate, device):
    wl = W.WORKLOADS["long32k"]
    k, N = wl.rates[rate]
    d, G, T, n_g = wl.d, wl.G, wl.T, wl.n_groups
    # the oracle's codebook, rounded to binary16 as the library's builder does
    R = oracle_rotation(d)
    C = quick_codebook(d, k, N).astype(np.float16).astype(np.float32)
    Rd, Cd = torch.from_numpy(R.copy()).to(device), torch.from_numpy(C.copy()).to(device)
    _say(f"[full size] long32k k={k} N={N}: {2 * n_g * T} vectors")
    kc = W.make_cache(wl, "k", device)
    vc = W.make_cache(wl, "v", device)
    q = W.group_view_query(W.make_query(wl, device), wl)
    kx, vx = kc.reshape(-1, d), vc.reshape(-1, d)
    n_v = kx.shape[0]
    kp, kn = fq.encode(kx, k, N, Rd, Cd)
    vp, vn = fq.encode(vx, k, N, Rd, Cd)
    torch.cuda.synchronize()

    rng = np.random.default_rng(100 + rate)
    rows = np.unique(np.concatenate([rng.integers(0, n_v, 3000), np.arange(64),
                                     np.arange(n_v - 64, n_v)]))
    ri = torch.from_numpy(rows).to(device)
    for name, x, p, nrm in (("K", kx, kp, kn), ("V", vx, vp, vn)):
        ne, nt, _, _ = gh.check_encode(gh.host_f64(x[ri]), R, C, N, p[ri], nrm[ri])
        _say(f"  encode {name}: {len(rows)} sampled rows, {ne} exact indices, {nt} near-ties")

    P = kp.shape[1]
    groups = [0, n_g // 2 + 3, n_g - 1]
    kpg, vpg = kp.view(n_g, T, P), vp.view(n_g, T, P)
    kng, vng = kn.view(n_g, T), vn.view(n_g, T)
    ref_pay = {}
    for g in groups:
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
