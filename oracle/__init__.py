"""CPU oracle of the tiered pooled-embedding lookup (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may load this module.  It wraps ``recmg_oracle.c`` (plain C,
built with gcc) through ctypes and shares no code with the HIP path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import tempfile
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "recmg_oracle.c")

FWD_FIELDS = ("lookups", "unique", "hits", "hits_prefetch", "misses", "ondemand_bytes", "prefetch_covered")
PLC_FIELDS = ("evicted", "admitted_miss", "prefetch_fill", "prefetch_resident",
              "prefetch_dropped", "miss_dropped", "resident", "prefetch_bytes", "prefetch_distinct")
DTYPES = {"f32": 0, "f16": 1, "bf16": 2}
POLICIES = {"lru": 0, "priority": 1, "lfu": 2}


def lib_path(mutant: int = 0) -> str:
    if mutant == 0:
        return os.path.join(HERE, "liboracle.so")
    d = os.path.join(tempfile.gettempdir(), "recmg_oracle_mutants")
    os.makedirs(d, exist_ok=True)
    return os.path.join(d, f"liboracle_mutant{mutant}.so")


def build(mutant: int = 0, out: Optional[str] = None) -> str:
    """Compile the oracle with gcc (``mutant`` > 0 plants a known mistake, for tests)."""
    out = out or lib_path(mutant)
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", f"-DORACLE_MUTANT={int(mutant)}",
           SRC, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_LIBS: dict = {}


def load(mutant: int = 0) -> ctypes.CDLL:
    lib = _LIBS.get(mutant)
    if lib is not None:
        return lib
    path = lib_path(mutant)
    if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(SRC):
        build(mutant)
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.oracle_create.restype = P
    lib.oracle_create.argtypes = [ctypes.c_int32, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_int32]
    lib.oracle_destroy.argtypes = [P]
    lib.oracle_placement.restype = ctypes.c_int32
    lib.oracle_placement.argtypes = [P, P, P, P]
    lib.oracle_forward.restype = ctypes.c_int32
    lib.oracle_forward.argtypes = [P, P, P, ctypes.c_int32, P, P]
    lib.oracle_table_stats.argtypes = [P, ctypes.c_int32, P, P, P]
    lib.oracle_resident.restype = ctypes.c_int64
    lib.oracle_resident.argtypes = [P, ctypes.c_int32, P, ctypes.c_int64]
    lib.oracle_pooled_abs.restype = ctypes.c_int32
    lib.oracle_pooled_abs.argtypes = [P, P, P, ctypes.c_int32, P]
    lib.oracle_splitmix64_mix.restype = ctypes.c_uint64
    lib.oracle_splitmix64_mix.argtypes = [ctypes.c_uint64]
    _LIBS[mutant] = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


class Oracle:
    """The tiered lookup and cache-state machine on the CPU.

    ``tables`` are numpy arrays [rows, dim] in storage type (float32, float16,
    or uint16 bfloat16 bits); they must stay alive as long as the oracle.
    ``ways`` = 0: fully associative caches; W > 0: W-way set-associative
    caches with Alg. 2 run inside each set."""

    def __init__(self, tables: Sequence[np.ndarray], dtypes: Sequence[str], caps: Sequence[int],
                 policy: str = "lru", eviction_speed: int = 4, nthreads: int = 1, mutant: int = 0,
                 ways: int = 0):
        self.lib = load(mutant)
        self.T = len(tables)
        self._tables = [np.ascontiguousarray(t) for t in tables]
        self.dims = [int(t.shape[1]) for t in self._tables]
        rows = np.array([t.shape[0] for t in self._tables], dtype=np.int64)
        dims = np.array(self.dims, dtype=np.int32)
        dts = np.array([DTYPES[d] for d in dtypes], dtype=np.int32)
        ptrs = (ctypes.c_void_p * self.T)(*[t.ctypes.data for t in self._tables])
        caps_a = np.array(caps, dtype=np.int64)
        self.h = self.lib.oracle_create(self.T, rows.ctypes.data, dims.ctypes.data, dts.ctypes.data,
                                        ctypes.cast(ptrs, ctypes.c_void_p), caps_a.ctypes.data,
                                        POLICIES[policy], int(eviction_speed), int(nthreads), int(ways))
        if not self.h:
            raise ValueError("oracle_create rejected the configuration")

    def close(self):
        if self.h:
            self.lib.oracle_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def placement(self, prefetch: np.ndarray, poff: np.ndarray, bits: Optional[np.ndarray] = None) -> int:
        prefetch = np.ascontiguousarray(prefetch, dtype=np.int32)
        poff = np.ascontiguousarray(poff, dtype=np.int64)
        bits = None if bits is None else np.ascontiguousarray(bits, dtype=np.uint8)
        if prefetch.size == 0:
            prefetch = np.zeros(1, np.int32)
        return int(self.lib.oracle_placement(self.h, _ptr(prefetch), _ptr(poff), _ptr(bits)))

    def forward(self, indices: np.ndarray, offsets: np.ndarray, bags: int, want64: bool = False,
                out32: Optional[np.ndarray] = None, out64: Optional[np.ndarray] = None):
        """Returns (status, out32 [sum_t B*D_t], out64 or None).  out32 / out64:
        caller-allocated outputs (float32 / float64, at least that size) to write
        instead of new arrays; out64 given implies want64."""
        indices = np.ascontiguousarray(indices, dtype=np.int32)
        offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        if indices.size == 0:
            indices = np.zeros(1, np.int32)
        n = bags * sum(self.dims)
        want64 = want64 or out64 is not None
        if out32 is None:
            out32 = np.zeros(max(n, 1), dtype=np.float32)
        if out64 is None and want64:
            out64 = np.zeros(max(n, 1), dtype=np.float64)
        assert out32.dtype == np.float32 and out32.size >= n and out32.flags.c_contiguous
        assert not want64 or (out64.dtype == np.float64 and out64.size >= n and out64.flags.c_contiguous)
        st = int(self.lib.oracle_forward(self.h, _ptr(indices), _ptr(offsets), int(bags), _ptr(out32), _ptr(out64)))
        return st, out32[:n], (out64[:n] if want64 else None)

    def pooled_abs(self, indices: np.ndarray, offsets: np.ndarray, bags: int) -> np.ndarray:
        """Per pooled output element, the sum of |x_i| over its bag (float64,
        table-major like forward's output): the tolerance scale.  Stateless."""
        indices = np.ascontiguousarray(indices, dtype=np.int32)
        offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        if indices.size == 0:
            indices = np.zeros(1, np.int32)
        n = bags * sum(self.dims)
        out = np.zeros(max(n, 1), dtype=np.float64)
        st = int(self.lib.oracle_pooled_abs(self.h, _ptr(indices), _ptr(offsets), int(bags), _ptr(out)))
        if st != 0:
            raise ValueError(f"oracle_pooled_abs returned {st}")
        return out[:n]

    def stats(self, t: int) -> dict:
        fwd = np.zeros(len(FWD_FIELDS), np.int64)
        plc = np.zeros(len(PLC_FIELDS), np.int64)
        dig = np.zeros(1, np.uint64)
        self.lib.oracle_table_stats(self.h, int(t), _ptr(fwd), _ptr(plc), _ptr(dig))
        d = {k: int(v) for k, v in zip(FWD_FIELDS, fwd)}
        d.update({k: int(v) for k, v in zip(PLC_FIELDS, plc)})
        d["digest"] = int(dig[0])
        return d

    def resident(self, t: int) -> np.ndarray:
        n = int(self.lib.oracle_resident(self.h, int(t), None, 0))
        out = np.zeros(max(n, 1), np.int32)
        self.lib.oracle_resident(self.h, int(t), _ptr(out), n)
        return out[:n]


def splitmix64_mix(z: int, mutant: int = 0) -> int:
    return int(load(mutant).oracle_splitmix64_mix(ctypes.c_uint64(z & ((1 << 64) - 1))))


def for_workload(w, tables: Sequence[np.ndarray], nthreads: int = 1, mutant: int = 0) -> Oracle:
    """An oracle configured like workload ``w`` (a ``tracegen.Workload``)."""
    return Oracle(tables, [tb.dtype for tb in w.tables], [tb.cap for tb in w.tables], policy=w.policy,
                  eviction_speed=w.eviction_speed, nthreads=nthreads, mutant=mutant, ways=w.ways)
