"""Shared, cached oracle objects for the tests (codebooks are slow to build)."""
import functools

import numpy as np

from oracle import codebook as ocb


@functools.lru_cache(maxsize=None)
def oracle_codebook(d, k, N, seed=1, M=None, restarts=4, iters=25):
    C, D = ocb.build_codebook(d, k, N, seed, M=M, restarts=restarts, iters=iters)
    C.setflags(write=False)
    return C, D


@functools.lru_cache(maxsize=None)
def oracle_rotation(d, seed=2):
    R = ocb.haar_rotation(d, seed).astype(np.float32)
    R.setflags(write=False)
    return R


def quick_codebook(d, k, N, seed=1):
    """A small-budget oracle codebook: any codebook serves for codec parity."""
    M = max(20 * N, 4000)
    return oracle_codebook(d, k, N, seed, M=M, restarts=1, iters=4)[0].astype(np.float32)


def read_table(path):
    rows = []
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows
