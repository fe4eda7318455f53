"""Benchmark of the FibQuant codec hot path on one MI355X.

A step is one pass of the whole hot path over one batch of the 32k-context
sub-one-bit workload (22 layers x 4 batch x 4 KV heads x 32768 tokens, d=64,
bf16 K and V, k=8, N=16, b=0.5, 32 query heads, GQA group 8):
  1. encode the K cache and the V cache (norm, rotation, nearest codeword,
     bit-packed 4-bit indices + fp16 norm);
  2. fused dequantisation + single-query decode attention over the whole
     compressed cache (all layers, batch rows and heads in one call);
  3. random-access decode of 65536 seeded token ids of the K cache.
Inputs are synthetic and resident in HBM before timing starts.  ``value`` is
the step's algorithmic bytes (encode: raw in + payload and norm out;
attention: compressed K+V, query, output; decode: payload, norm, id in,
fp32 rows out) per second.  One JSON line is printed.
"""
import argparse
import dataclasses
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2605_11478_amd as fq  # noqa: E402
from paper_2605_11478_amd import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, 8 TB/s
N_DECODE = 65536
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def measured_traffic(kernel, workload, rate):
    """HBM bytes per launch of `kernel` from the committed counter record
    (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by what the same
    counter reads for a 1 GiB device copy), or None when the record is
    missing, was taken on another workload, or the kernel's source has
    changed since it was taken."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        k = rec["kernels"][kernel]
        if rec["workload"] != workload or rec["rate"] != rate:
            return None
        src = os.path.join(ROOT, k["source"])
        with open(src, "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != k["sha256"]:
                return None
        cal = rec["calibration"]
        return round(1024 * (k["fetch_kib"] * cal["read_factor"] + k["write_kib"] * cal["write_factor"]))
    except (OSError, KeyError, ValueError):
        return None


MFMA_F16_PEAK_TFLOPS = 2500.0   # MI355X dense fp16 / bf16 matrix peak
COLD_COPIES = 6                 # copies of the compressed cache cycled by the cold attention
COLD_LAUNCHES = 60              # timed cold attention launches (at least)
COLD_WARMUP = 120               # untimed attention launches before them
SETTLE_S = 0.25                 # seconds of untimed steps after the W warm-up steps


def spread(ms):
    """Launch durations (ms): count, mean, median, 10th and 90th percentile."""
    v = np.asarray(ms, dtype=np.float64)
    return {"n": int(v.size), "mean": round(float(v.mean()), 4),
            "median": round(float(np.median(v)), 4),
            "p10": round(float(np.percentile(v, 10)), 4),
            "p90": round(float(np.percentile(v, 90)), 4)}


def encode_roofline(enc_bytes, enc_flops, enc_ms, workload, rate):
    gbs = enc_bytes / (enc_ms * 1e-3) / 1e9
    if enc_flops / enc_bytes <= MFMA_F16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        return {"bound": "hbm", "kernel": "encode (one cache per launch)",
                "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("encode", workload, rate)}
    tf = enc_flops / (enc_ms * 1e-3) / 1e12
    return {"bound": "mfma", "kernel": "encode (one cache per launch)",
            "achieved": round(tf, 3), "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tf / MFMA_F16_PEAK_TFLOPS, 4),
            "traffic": measured_traffic("encode", workload, rate)}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="long32k")
    ap.add_argument("--rate", type=int, default=0, help="index into the workload's (k, N) list")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--all-workloads", action="store_true",
                    help="one JSON line per workload and rate (no CPU baseline), after the default line")
    ap.add_argument("--radius-first", action="store_true",
                    help="also time the radius-first encoder (App. F Stage 1) against the "
                         "exhaustive one on multi-shell codebooks, with the NMSE of each")
    ap.add_argument("--rate-axis", action="store_true",
                    help="one JSON line per (k, N) point of the paper's rate axis on the GPT-2-shaped "
                         "cache (no CPU baseline), after the default line")
    return ap.parse_args()


def host_info():
    """Logical CPUs visible to this process, the CPU model and the BLAS thread
    count of the NumPy that runs the oracle."""
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        blas = 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"nproc": usable, "cpu_count": os.cpu_count(), "cpu_model": model,
            "blas_threads": int(blas)}


def cpu_baseline(wl, k, N, R, C, kx, vx, q, budget_s=12.0, max_groups=128):
    """The oracle, untuned, on a bounded sample of the same workload: whole
    (layer, batch, KV head) groups in order, each encoded (K and V, packed)
    and attended from its payload, until ``budget_s`` of oracle time has
    passed (at most ``max_groups`` groups).  Encode and attention are timed
    separately: encode vectors/s, attention cache tokens/s and the GB/s each
    implies, plus the whole sample's GB/s counted as ``value`` counts bytes."""
    from oracle import attention as oat
    from oracle import codec as occ
    info = host_info()
    d, T = wl.d, wl.T
    # groups whose oracle encode would take minutes (large N) are cut to a token prefix
    Tg = T if T * d * N <= 2 ** 32 else max(1024, 2 ** 32 // (d * N))
    R64, C64 = R.astype(np.float64), C.astype(np.float64)
    P = fq.payload_bytes(d, k, N)
    rows = max(1, 2 ** 25 // ((d // k) * N))  # rows per oracle call (its D is rows x d/k x N)

    def enc(xg):
        parts = [occ.encode(xg[s:s + rows], R64, C64) for s in range(0, len(xg), rows)]
        return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])

    in_b = kx.element_size()
    t_enc = t_att = 0.0
    groups = 0
    while t_enc + t_att < budget_s and groups < min(max_groups, wl.n_groups):
        g = groups
        kg = kx[g * T:g * T + Tg].double().cpu().numpy()  # host copies: not timed
        vg = vx[g * T:g * T + Tg].double().cpu().numpy()
        qg = q[g].double().cpu().numpy()
        t0 = time.perf_counter()
        ki, kh = enc(kg)
        vi, vh = enc(vg)
        kpay, vpay = occ.pack(ki, N), occ.pack(vi, N)
        t1 = time.perf_counter()
        o = oat.attention_from_payload(qg, kpay, occ.fp16_bits(kh), vpay, occ.fp16_bits(vh),
                                       R64, C64, N)
        t2 = time.perf_counter()
        t_enc += t1 - t0
        t_att += t2 - t1
        groups += 1
    assert np.isfinite(o).all()
    secs = t_enc + t_att
    enc_bytes = 2 * Tg * (d * in_b + P + 2)
    attn_bytes = 2 * Tg * (P + 2) + wl.G * d * (q.element_size() + 4)
    return {"value": round(groups * (enc_bytes + attn_bytes) / secs / 1e9, 6), "unit": "GB/s",
            "cores": info["blas_threads"], "kind": "oracle",
            "sample": (f"float64 NumPy oracle on {groups} of the {wl.n_groups} groups (each: "
                       f"encode + pack {Tg} K and {Tg} V vectors, decode from the payload, naive "
                       f"attention of G={wl.G} heads); {secs:.1f} s; bytes counted as in value; "
                       f"matrix products on {info['blas_threads']} BLAS threads, the rest of "
                       f"the oracle on one core"),
            "seconds": round(secs, 2),
            "encode": {"vectors_per_s": round(2 * Tg * groups / t_enc, 1),
                       "GB_per_s": round(groups * enc_bytes / t_enc / 1e9, 6),
                       "seconds": round(t_enc, 2)},
            "attention": {"cache_tokens_per_s": round(Tg * groups / t_att, 1),
                          "GB_per_s": round(groups * attn_bytes / t_att / 1e9, 6),
                          "seconds": round(t_att, 2)},
            "host": info}


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); the codec has no "
              "multi-GPU path; run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    print(json.dumps(run(a, a.workload, a.rate, not a.no_cpu_baseline)), flush=True)
    if a.all_workloads:
        for name, wl in W.WORKLOADS.items():
            for rate in range(len(wl.rates)):
                if (name, rate) == (a.workload, a.rate):
                    continue
                torch.cuda.empty_cache()
                print(json.dumps(run(a, name, rate, False)), flush=True)
    if a.radius_first:
        for name, L in RADIUS_FIRST:
            torch.cuda.empty_cache()
            print(json.dumps(radius_first_run(a, name, L)), flush=True)
    if a.rate_axis:
        for k, N in RATE_AXIS:
            torch.cuda.empty_cache()
            wl = dataclasses.replace(W.WORKLOADS["gpt2"], rates=((k, N),))
            print(json.dumps(run(a, wl, 0, False, quick_codebook=True)), flush=True)


# workloads and shell counts (L = sqrt(N)) for the radius-first encoder
RADIUS_FIRST = [("gpt2", 16), ("tinyllama", 16), ("stress", 64)]


def radius_first_run(a, name, L):
    """Radius-first encoder (App. F Stage 1), list decoding inside the shell
    (Stages 1 + 2) and the exhaustive encoder on one cache of a workload, all
    with the same multi-shell codebook C(L, N/L) (two Lloyd rounds): per-cache
    encode time and the NMSE of the decoded cache (the price of the
    approximate searches)."""
    dev = "cuda:0"
    wl = W.WORKLOADS[name]
    k, N = wl.rates[0]
    d = wl.d
    R = fq.build_rotation(d, wl.rotation_seed)
    C, _ = fq.build_codebook(d, k, N, wl.codebook_seed, M=max(4000, 4 * N), restarts=1, iters=2,
                             init="multishell", shells=L)
    Rd, Cd = torch.from_numpy(R).to(dev), torch.from_numpy(C).to(dev)
    x = W.make_cache(wl, "k", dev).reshape(-1, d)
    n_v = x.shape[0]
    P = fq.payload_bytes(d, k, N)
    pay = torch.empty((n_v, P), dtype=torch.uint8, device=dev)
    nrm = torch.empty((n_v,), dtype=torch.int16, device=dev)
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(a.warmup):
            fn()
        evs = []
        for _ in range(a.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            evs.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.mean([e0.elapsed_time(e1) for e0, e1 in evs]))

    def nmse_db():  # on a fixed sample of 65536 rows, decoded on the device
        ids = torch.randint(0, n_v, (N_DECODE,), generator=torch.Generator().manual_seed(5)).to(dev)
        xh = fq.decode(pay, nrm, d, k, N, Rd, Cd, token_ids=ids)
        xs = x[ids].float()
        return float(10 * torch.log10(((xs - xh) ** 2).sum() / (xs * xs).sum()))

    ms_rf = timed(lambda: fq.encode_radius_first(x, k, N, L, Rd, Cd, pay, nrm))
    db_rf = nmse_db()
    # Stage 2 inside the shell: K ~ sqrt(T M_a) parents, the best T = 2 searched
    Kp, Tl = (4, 2) if N // L <= 16 else (8, 2)
    mu, off, mem = fq.build_parent_lists(C, L, Kp)
    mud, offd, memd = (torch.from_numpy(a).to(dev) for a in (mu, off, mem))
    ms_ls = timed(lambda: fq.encode_list(x, k, N, L, Kp, Tl, mud, offd, memd, Rd, Cd, pay, nrm))
    db_ls = nmse_db()
    ms_ex = timed(lambda: fq.encode(x, k, N, Rd, Cd, pay, nrm))
    db_ex = nmse_db()
    in_bytes = n_v * (d * x.element_size() + P + 2)
    gbs = in_bytes / (ms_rf * 1e-3) / 1e9
    return {"metric": "radius-first encode GB/s (App. F Stage 1), one cache",
            "value": round(gbs, 3), "unit": "GB/s", "frac_hbm": round(gbs / 8000.0, 4),
            "dtype": str(x.dtype).replace("torch.", ""),
            "config": {"workload": f"{name}: {n_v} vectors, d={d}, k={k}, N={N}, L={L} shells "
                                   f"of {N // L}"},
            "encode_ms": {"radius_first": round(ms_rf, 4), f"list_K{Kp}_T{Tl}": round(ms_ls, 4),
                          "exhaustive": round(ms_ex, 4)},
            "speedup": round(ms_ex / ms_rf, 2),
            "nmse_db": {"radius_first": round(db_rf, 3), f"list_K{Kp}_T{Tl}": round(db_ls, 3),
                        "exhaustive": round(db_ex, 3)}}


# (k, N) points of the paper's rate axis (its GPT-2 study: scalar k = 1, the
# vector codes at b = 3 .. 0.75 and the large-block codes down to b = 0.22)
RATE_AXIS = [(1, 4), (1, 16), (2, 64), (4, 256), (8, 256), (8, 1024), (8, 4096), (16, 4096),
             (32, 16384), (64, 16384)]


def run(a, workload, rate, with_cpu, quick_codebook=False):
    dev = "cuda:0"
    wl = W.WORKLOADS[workload] if isinstance(workload, str) else workload
    k, N = wl.rates[rate]
    d, G, T, n_g = wl.d, wl.G, wl.T, wl.n_groups
    P = fq.payload_bytes(d, k, N)

    R = fq.build_rotation(d, wl.rotation_seed)
    if quick_codebook and k == d:
        # the full-vector code: the unpolished construction (its 4 MB codebook
        # would take minutes of host Lloyd; throughput does not depend on it)
        C, _ = fq.build_codebook(d, k, N, wl.codebook_seed, M=4000, restarts=1, iters=0)
    elif quick_codebook:  # a small Lloyd budget: throughput does not depend on the polish
        C, _ = fq.build_codebook(d, k, N, wl.codebook_seed, M=max(4000, 4 * N), restarts=1, iters=2)
    else:
        C, _ = fq.build_codebook(d, k, N, wl.codebook_seed)
    Rd, Cd = torch.from_numpy(R).to(dev), torch.from_numpy(C).to(dev)

    kc = W.make_cache(wl, "k", dev)
    vc = W.make_cache(wl, "v", dev)
    q = W.group_view_query(W.make_query(wl, dev), wl)
    kx, vx = kc.reshape(-1, d), vc.reshape(-1, d)
    n_v = kx.shape[0]
    kp = torch.empty((n_v, P), dtype=torch.uint8, device=dev)
    vp = torch.empty((n_v, P), dtype=torch.uint8, device=dev)
    kn = torch.empty((n_v,), dtype=torch.int16, device=dev)
    vn = torch.empty((n_v,), dtype=torch.int16, device=dev)
    ws = torch.zeros((fq.attn_workspace_bytes(n_g, G, T, d, k, N),), dtype=torch.uint8,
                     device=dev)
    out = torch.empty((n_g, G, d), dtype=torch.float32, device=dev)
    ids = torch.randint(0, n_v, (N_DECODE,), generator=torch.Generator().manual_seed(11)).to(dev)
    xh = torch.empty((N_DECODE, d), dtype=torch.float32, device=dev)

    stream = torch.cuda.current_stream()
    ev = {n: [] for n in ("enc_k", "enc_v", "attn", "dec")}

    def attend(kp_, kn_, vp_, vn_):
        fq.attn_decode(q, kp_.view(n_g, T, P), kn_.view(n_g, T), vp_.view(n_g, T, P),
                       vn_.view(n_g, T), T, k, N, Rd, Cd, workspace=ws, out=out)

    def step(record):
        marks = []
        def mark():
            if record:
                e = torch.cuda.Event(enable_timing=True)
                e.record(stream)
                marks.append(e)
        mark()
        fq.encode(kx, k, N, Rd, Cd, kp, kn)
        mark()
        fq.encode(vx, k, N, Rd, Cd, vp, vn)
        mark()
        attend(kp, kn, vp, vn)
        mark()
        fq.decode(kp, kn, d, k, N, Rd, Cd, token_ids=ids, out=xh)
        mark()
        if record:
            for i, n in enumerate(("enc_k", "enc_v", "attn", "dec")):
                ev[n].append((marks[i], marks[i + 1]))

    for _ in range(a.warmup):
        step(False)
    torch.cuda.synchronize()
    # Untimed clock settling: the shader clock climbs for the first ~50 ms of
    # sustained encoder work (per-launch encode time falls by ~10 %), so
    # warm-up continues until SETTLE_S seconds have passed, whatever W is.
    settle_steps, t_s = 0, time.perf_counter()
    while time.perf_counter() - t_s < SETTLE_S:
        step(False)
        settle_steps += 1
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        step(True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    # The fused attention alone, with the compressed cache out of the 256 MB
    # Infinity Cache: launches cycle over COLD_COPIES device copies of it
    # (each read again only after the other copies' bytes have streamed), so
    # every launch reads its payload from HBM.  Not part of the step time.
    copies = [(kp.clone(), kn.clone(), vp.clone(), vn.clone()) for _ in range(COLD_COPIES)]
    for i in range(COLD_WARMUP):  # untimed: the clocks settle after the encode-heavy steps
        attend(*copies[i % COLD_COPIES])
    cold = []
    for i in range(max(a.steps, COLD_LAUNCHES)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        attend(*copies[i % COLD_COPIES])
        e1.record(stream)
        cold.append((e0, e1))
    torch.cuda.synchronize()
    del copies
    if a.copy_calibration and (workload, rate) == (a.workload, a.rate):
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
    times = {n: [s_.elapsed_time(e_) for s_, e_ in v] for n, v in ev.items()}
    times["enc"] = times["enc_k"] + times["enc_v"]
    times["attn_cold"] = [s_.elapsed_time(e_) for s_, e_ in cold]
    ms = {n: float(np.mean(v)) for n, v in times.items()}
    in_b = kx.element_size()
    enc_bytes = n_v * (d * in_b + P + 2)
    enc_flops = n_v * (2 * d * d + 2 * d * N + 2 * d)
    attn_bytes = 2 * n_g * T * (P + 2) + n_g * G * d * (q.element_size() + 4)
    dec_bytes = N_DECODE * (P + 2 + 8 + 4 * d)
    step_bytes = 2 * enc_bytes + attn_bytes + dec_bytes
    ms_step = elapsed * 1e3 / a.steps
    enc_ms = ms["enc"]
    attn_ms = ms["attn_cold"]
    attn_gbs = attn_bytes / (attn_ms * 1e-3) / 1e9
    enc_gbs = enc_bytes / (enc_ms * 1e-3) / 1e9
    enc_tflops = enc_flops / (enc_ms * 1e-3) / 1e12
    res = {
        "metric": "KV encode GB/s + fused dequant-attention decode GB/s, % of HBM peak",
        "value": round(step_bytes / (ms_step * 1e-3) / 1e9, 3),
        "unit": "GB/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "settle_steps": settle_steps,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16/fp16 mfma, fp32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: {wl.layers} layers x {wl.batch} batch x {wl.kv_heads} "
                         f"KV heads x {T} tokens, d={d}, {str(wl.dtype).split('.')[-1]} K/V, "
                         f"{wl.q_heads} query heads (G={G}); k={k}, N={N}, "
                         f"b={math.log2(N) / k:g} bits/coord"),
            "step": "encode K + encode V + fused attention over all groups + decode of "
                    f"{N_DECODE} token ids",
            "cache_vectors": 2 * n_v, "compressed_cache_bytes": 2 * n_v * (P + 2),
        },
        "encode": {"ms": round(enc_ms, 4), "GB_per_s": round(enc_gbs, 2),
                   "frac_hbm": round(enc_gbs / HBM_PEAK_GBS, 4),
                   "TFLOP_per_s": round(enc_tflops, 3),
                   "vectors_per_s": round(n_v / (enc_ms * 1e-3), 1),
                   "launch_ms": spread(times["enc"])},
        "attention": {"ms": round(attn_ms, 4), "GB_per_s": round(attn_gbs, 2),
                      "frac_hbm": round(attn_gbs / HBM_PEAK_GBS, 4),
                      "cache_tokens_per_s": round(n_g * T / (attn_ms * 1e-3), 1),
                      "decode_steps_per_s": round(1e3 / attn_ms, 2),
                      "launch_ms": spread(times["attn_cold"]),
                      "cache": (f"out of the Infinity Cache: launches cycle over {COLD_COPIES} "
                                f"device copies of the compressed cache "
                                f"({COLD_COPIES * 2 * n_v * (P + 2) / 1e9:.2f} GB)"),
                      "in_step_ms": spread(times["attn"])},
        "decode": {"ms": round(ms["dec"], 4),
                   "GB_per_s": round(dec_bytes / (ms["dec"] * 1e-3) / 1e9, 2),
                   "launch_ms": spread(times["dec"])},
        # dominant kernel: the encoder (two launches per step).  Its roof is HBM
        # (d * in + P + 2 algorithmic bytes per vector) unless its algorithmic
        # intensity (2 d^2 + 2 d N + 2 d flops per vector) exceeds the fp16
        # matrix-core ridge, as for N = 4096; then it is the fp16 MFMA peak.
        "roofline": encode_roofline(enc_bytes, enc_flops, enc_ms, wl.name, rate),
        "roofline_attention": {"bound": "hbm", "kernel": "fused attention (one call, all groups)",
                               "achieved": round(attn_gbs, 2), "peak": HBM_PEAK_GBS,
                               "unit": "GB/s", "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                               "traffic": measured_traffic("attention", wl.name, rate)},
    }
    if with_cpu:
        res["cpu_baseline"] = cpu_baseline(wl, k, N, R, C, kx, vx, q)
    return res


if __name__ == "__main__":
    main()
