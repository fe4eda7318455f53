"""Summarise two rocprofv3 counter passes of ``bench.py`` into
``profiles/traffic.json`` (the HBM bytes ``bench.py`` reports as
``roofline.traffic``).

Usage, after running from the repository root on an MI355X::

    rocprofv3 --pmc FETCH_SIZE -d <fetch_dir> -o run --output-format csv -- \
        python -u bench.py --steps 2 --warmup 0 --no-cpu-baseline --copy-calibration
    rocprofv3 --pmc WRITE_SIZE -d <write_dir> -o run --output-format csv -- \
        python -u bench.py --steps 2 --warmup 0 --no-cpu-baseline --copy-calibration
    python -m paper_2605_11478_amd.traffic <fetch_dir> <write_dir>

Both counters are in KiB per dispatch.  ``--copy-calibration`` makes the bench
run one 1 GiB device-to-device copy after the timed steps; what the counters
read for that copy (1 GiB read, 1 GiB written) gives the factor each counter
is scaled by.  A kernel's figure is the mean over its dispatches; the
attention entry sums the kernels of one attention launch.  Each entry records
the SHA-256 of the source its kernels are built from, so that ``bench.py``
stops reporting it once that source changes.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_KERNEL = "__amd_rocclr_copyBuffer"
GIB_KIB = 1024.0 * 1024.0

# entry -> (source file, kernel-name fragments of one launch)
KERNELS = {
    "encode": ("paper_2605_11478_amd/csrc/encode_mfma.hip", ["encmf::encode_kernel"]),
    "attention": ("paper_2605_11478_amd/csrc/attn_w4.hip",
                  ["w4::main_kernel", "w4::merge_kernel"]),
}


def _read(d, counter):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    per = defaultdict(float)  # (kernel, dispatch) -> value
    for fn in files:
        with open(fn) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter:
                    per[(r["Kernel_Name"], r["Dispatch_Id"])] += float(r["Counter_Value"])
    by_kernel = defaultdict(list)
    for (name, _), v in per.items():
        by_kernel[name].append(v)
    return by_kernel


def _match(by_kernel, frag):
    # rocprofv3 reports some names demangled and some mangled: "ns::kern"
    # appears in the mangled form as "2ns4kern"
    mangled = "".join(f"{len(p)}{p}" for p in frag.split("::"))
    hits = [v for name, v in by_kernel.items() if frag in name or mangled in name]
    if len(hits) != 1:
        raise SystemExit(f"{len(hits)} kernels match {frag!r}")
    return sum(hits[0]) / len(hits[0])


def summarise(fetch_dir, write_dir, workload="long32k", rate=0):
    fetch, write = _read(fetch_dir, "FETCH_SIZE"), _read(write_dir, "WRITE_SIZE")
    # the calibration copy is the largest copy dispatch of the run
    cf, cw = max(fetch[COPY_KERNEL]), max(write[COPY_KERNEL])
    rec = {
        "note": ("FETCH_SIZE / WRITE_SIZE in KiB per dispatch (rocprofv3 --pmc, one counter "
                 "per pass), averaged over the dispatches of bench.py --steps 2 --warmup 0 "
                 "--no-cpu-baseline --copy-calibration; the attention entry sums the kernels "
                 "of one attention launch"),
        "workload": workload, "rate": rate,
        "calibration": {"kernel": COPY_KERNEL + ", 1 GiB device-to-device copy",
                        "fetch_kib": round(cf, 1), "write_kib": round(cw, 1),
                        "read_factor": round(GIB_KIB / cf, 3),
                        "write_factor": round(GIB_KIB / cw, 3)},
        "kernels": {},
    }
    for name, (src, frags) in KERNELS.items():
        with open(os.path.join(ROOT, src), "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
        parts = {fr: (_match(fetch, fr), _match(write, fr)) for fr in frags}
        rec["kernels"][name] = {
            "source": src, "sha256": sha, "kernel_name": " + ".join(frags),
            "fetch_kib": round(sum(p[0] for p in parts.values()), 1),
            "write_kib": round(sum(p[1] for p in parts.values()), 1),
            "parts": {fr: {"fetch_kib": round(p[0], 1), "write_kib": round(p[1], 1)}
                      for fr, p in parts.items()},
        }
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("fetch_dir")
    ap.add_argument("write_dir")
    ap.add_argument("--workload", default="long32k")
    ap.add_argument("--rate", type=int, default=0)
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "traffic.json"))
    a = ap.parse_args()
    rec = summarise(a.fetch_dir, a.write_dir, a.workload, a.rate)
    with open(a.out, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    main()
