"""Parity at full workload sizes, in the launch configuration the benchmark
times: one encode call per cache and one attention call over all groups
(many token units per wavefront, groups shared between workgroups).  The
float64 oracle cannot encode whole caches of tens of millions of vectors, so
it checks sampled outputs it computes one by one:

  * encode: seeded random rows plus the first and last 64 rows of each cache
    (indices up to the near-tie rule, payload bytes and header bits);
  * attention: three whole groups (first, a middle one, last).  Where the
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
    groups = [0, n_g // 2 + 3, n_g - 1]
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
