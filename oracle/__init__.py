"""Plain CPU oracle for the FibQuant random-access KV-cache codec.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything in this package; only
the test-suite, the smoke check and the CPU-baseline leg of the benchmark do.

Everything here is written from the paper (arXiv 2605.11478, "FibQuant:
Universal Vector Quantization for Random-Access KV-Cache Compression") in
float64 NumPy, as slowly and plainly as possible, so that a reader can check
each function against the cited section or equation by eye:

* ``philox``    counter-based generator (Salmon et al., SC'11) + Box-Muller
                normals; the published definition, implemented independently
                of the C++ one in the library.
* ``codebook``  Haar rotation, spherical-Beta sampler (Lemma 1), Beta-quantile
                radii (Eqs. radii_main / radii_k2), direction sets (Sec. 3.3,
                App. E) and the multi-restart Lloyd-Max polish (App. A table).
* ``codec``     norm header, rotation, per-block brute-force argmin
                (Eq. encode), fixed-width bit packing, decoder (Sec. 3.1).
* ``attention`` naive single-query softmax attention (Eq. lattn).
* ``fileio``    reader/writer of the codebook file format.
"""
