"""Shared test helpers: golden-file loading and run drivers (no method arithmetic)."""
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def golden_table(g):
    """Table values E[r][k] = r + 100*k (float32) of a hand-worked example."""
    r = np.arange(g["rows"], dtype=np.float32)[:, None]
    k = np.arange(g["dim"], dtype=np.float32)[None, :]
    return np.ascontiguousarray(r + 100.0 * k, dtype=np.float32)


def splitmix64_mix_py(z):
    """SplitMix64 output mix (Steele, Lea & Flood 2014) in Python integers."""
    m = (1 << 64) - 1
    z &= m
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return z ^ (z >> 31)


def l1_mass(tables_f64, dims, indices, offsets, bags):
    """Per output element, the sum of |x_i| over the bag (the tolerance scale)."""
    T = len(tables_f64)
    out = []
    for t in range(T):
        tab = np.abs(tables_f64[t])
        for j in range(bags):
            a, e = offsets[t * bags + j], offsets[t * bags + j + 1]
            out.append(tab[indices[a:e]].sum(axis=0) if e > a else np.zeros(dims[t]))
    return np.concatenate(out) if out else np.zeros(0)
