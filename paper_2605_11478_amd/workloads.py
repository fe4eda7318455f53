"""Seeded synthetic KV-cache workloads.

This module holds only shapes and seeded random inputs; none of the codec's
arithmetic lives here.  Both the GPU path (tests, benchmark) and the CPU
oracle (tests) draw their inputs from it.

The caches stand in for the KV caches of the paper's GPT-2-small and
TinyLlama-1.1B experiments (Sec. 5.2, 5.3), whose model weights and datasets
are not used here.  Element laws:

* ``normal``: x ~ N(0, 1) (the small fp32 case);
* ``lognormal_outlier``: x = sigma_c * N(0, 1) per channel c, with
  sigma_c ~ LogNormal(0, 0.5) drawn per (layer, kv-head, channel) and two
  channels per (layer, kv-head), chosen by a seeded permutation, scaled by
  10 (outlier channels); drawn independently for K and V.

Queries are N(0, 1) in the cache dtype (fp32 for the small case).
Seeds: base = 1000 * workload number (0 for the small case); K data base+0,
V data base+5, query base+3, sigma/outliers base+4 (K) and base+9 (V).
"""
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    number: int
    layers: int
    batch: int
    kv_heads: int
    q_heads: int
    T: int
    d: int
    dtype: torch.dtype
    law: str
    rates: tuple  # ((k, N), ...)
    codebook_seed: int = 1
    rotation_seed: int = 2

    @property
    def G(self):
        return self.q_heads // self.kv_heads

    @property
    def n_groups(self):
        return self.layers * self.batch * self.kv_heads

    @property
    def n_vec(self):
        """Vectors per cache (K or V)."""
        return self.n_groups * self.T

    @property
    def base_seed(self):
        return 1000 * self.number


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 1, 1, 1, 4096, 64, torch.float32, "normal", ((2, 16),)),
    "gpt2": Workload("gpt2", 1, 12, 1, 12, 12, 1024, 64, torch.float16, "lognormal_outlier",
                     ((4, 256),)),
    "tinyllama": Workload("tinyllama", 2, 22, 8, 4, 32, 2048, 64, torch.bfloat16,
                          "lognormal_outlier", ((4, 256), (2, 64))),
    "long32k": Workload("long32k", 3, 22, 4, 4, 32, 32768, 64, torch.bfloat16,
                        "lognormal_outlier", ((8, 16), (8, 64))),
    "stress": Workload("stress", 4, 32, 1, 8, 32, 131072, 128, torch.bfloat16,
                       "lognormal_outlier", ((4, 4096),)),
}


def _gen(seed, device):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def channel_sigma(wl, which):
    """Per (layer, kv-head, channel) std-devs [layers, kv_heads, d] (float32, CPU)."""
    if wl.law == "normal":
        return torch.ones(wl.layers, wl.kv_heads, wl.d)
    seed = wl.base_seed + (4 if which == "k" else 9)
    g = _gen(seed, "cpu")
    sig = torch.exp(0.5 * torch.randn(wl.layers, wl.kv_heads, wl.d, generator=g))
    for l in range(wl.layers):
        for h in range(wl.kv_heads):
            ch = torch.randperm(wl.d, generator=g)[:2]
            sig[l, h, ch] *= 10.0
    return sig


def make_cache(wl, which, device="cpu", T=None, layers=None):
    """K (``which='k'``) or V cache [layers, batch, kv_heads, T, d] in wl.dtype.

    ``T``/``layers`` shrink the cache for small tests (same law, same seeds).
    """
    T = wl.T if T is None else T
    L = wl.layers if layers is None else layers
    sig = channel_sigma(wl, which)[:L].to(device)
    g = _gen(wl.base_seed + (0 if which == "k" else 5), device)
    out = torch.empty(L, wl.batch, wl.kv_heads, T, wl.d, dtype=wl.dtype, device=device)
    for l in range(L):
        z = torch.randn(wl.batch, wl.kv_heads, T, wl.d, generator=g, device=device)
        z.mul_(sig[l][None, :, None, :])
        out[l].copy_(z)
        del z
    return out


def make_query(wl, device="cpu", layers=None):
    """Decode query [layers, batch, q_heads, d] in wl.dtype (q-head h uses kv-head h // G)."""
    L = wl.layers if layers is None else layers
    g = _gen(wl.base_seed + 3, device)
    q = torch.randn(wl.layers, wl.batch, wl.q_heads, wl.d, generator=g, device=device)
    return q[:L].to(wl.dtype).contiguous()


def group_view_query(q, wl):
    """[L, B, q_heads, d] -> [L*B*kv_heads, G, d] (the library's group layout)."""
    L = q.shape[0]
    return q.reshape(L, wl.batch, wl.kv_heads, wl.G, wl.d).reshape(-1, wl.G, wl.d)
