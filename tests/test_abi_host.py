"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/recmg.h declares, and recmg_query_workspace validates
configurations."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2511_08568_amd as pk
from paper_2511_08568_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "recmg.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int32_t|const char \*)\s*(recmg_\w+)\s*\(", src, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    assert names == sorted(bd.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = pk.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert isinstance(pk.recmg_last_error(), str)


def _cfg(rows=(1000,), dims=(64,), dtypes=(0,), caps=(100,), policy=0, miss=0, max_idx=5000, max_pf=5000,
         bags=256, es=4, ways=0):
    T = len(rows)
    keep = []
    cfg = bd.recmg_config_t()
    cfg.num_tables = T
    for name, ctype, vals in (("rows", ctypes.c_int64, rows), ("dims", ctypes.c_int32, dims),
                              ("dtypes", ctypes.c_int32, dtypes), ("cache_rows", ctypes.c_int64, caps)):
        arr = (ctype * T)(*vals)
        keep.append(arr)
        setattr(cfg, name, arr)
    bufs = [np.zeros(16 * r * d + 64, np.uint8) for r, d in zip(rows, dims)]
    ptrs = (ctypes.c_void_p * T)(*[(b.ctypes.data + 15) // 16 * 16 for b in bufs])
    keep += [bufs, ptrs]
    cfg.host_tables = ptrs
    cfg.policy, cfg.miss_mode, cfg.eviction_speed = policy, miss, es
    cfg.max_indices, cfg.max_prefetch, cfg.max_bags_per_table = max_idx, max_pf, bags
    cfg.ways = ways
    cfg._keep = keep
    return cfg


def test_query_workspace_sizes():
    dev, host = bd.recmg_query_workspace(_cfg())
    # at least the slot pool, its map and the staging rows
    assert dev >= 100 * 256 + 256 * 8 + 5000 * 256
    assert host == 0
    dev2, host2 = bd.recmg_query_workspace(_cfg(miss=1))
    # STAGED adds an HBM area for host-staged prefetch rows; pinned staging holds
    # miss rows and prefetch rows
    assert dev2 - dev >= 5000 * 256 - 256 and host2 >= 2 * 5000 * 256


def test_lfu_keeps_a_counter_per_row():
    """LFU_BATCH counts batches for every row: 4 bytes per row more workspace
    than PRIORITY, which keeps no per-row state."""
    prio, _ = bd.recmg_query_workspace(_cfg(rows=(100000,), policy=1))
    lfu, _ = bd.recmg_query_workspace(_cfg(rows=(100000,), policy=2))
    assert lfu - prio >= 4 * 100000 - 1024  # up to a few 256-byte alignments


def test_lru_keeps_a_resident_ring():
    """LRU_BATCH fully associative tables keep their residents in key order:
    two ring buffers of at least Cap + 3 x (max_indices + max_prefetch)
    entries, a slot -> entry index, the zones and the pending lists.  Tables
    with Cap 0 and set-associative tables keep none."""
    lru, _ = bd.recmg_query_workspace(_cfg(caps=(100,)))
    prio, _ = bd.recmg_query_workspace(_cfg(caps=(100,), policy=1))
    ring = 2 * 4 * (100 + 3 * (5000 + 5000))
    assert lru - prio >= ring + 8 * (5000 + 5000)
    lru0, _ = bd.recmg_query_workspace(_cfg(caps=(0,)))
    prio0, _ = bd.recmg_query_workspace(_cfg(caps=(0,), policy=1))
    assert lru0 - prio0 < 4096
    lru_sa, _ = bd.recmg_query_workspace(_cfg(caps=(128,), ways=32))
    prio_sa, _ = bd.recmg_query_workspace(_cfg(caps=(128,), ways=32, policy=1))
    assert lru_sa - prio_sa < 4096


def test_query_scales_with_capacity():
    a, _ = bd.recmg_query_workspace(_cfg(caps=(100,)))
    b, _ = bd.recmg_query_workspace(_cfg(caps=(1000,)))
    assert b - a >= 900 * 256


@pytest.mark.parametrize("kw", [dict(rows=(0,)), dict(dims=(0,)), dict(dtypes=(7,)), dict(caps=(-1,)),
                                dict(policy=5), dict(policy=3), dict(miss=9), dict(max_idx=-1), dict(es=-1),
                                dict(max_idx=1 << 31), dict(ways=-1), dict(ways=65)])
def test_query_rejects_bad_configs(kw):
    with pytest.raises(bd.RecmgError) as e:
        bd.recmg_query_workspace(_cfg(**kw))
    assert e.value.code == bd.RECMG_E_INVALID
    assert pk.recmg_last_error()


def test_set_associative_slots():
    """W-way sets use floor(Cap / W) * W slots: Cap 96, 100 and 127 all give 3
    sets of 32 (the same workspace), Cap 128 gives 4."""
    q = lambda cap: bd.recmg_query_workspace(_cfg(caps=(cap,), rows=(100000,), ways=32))[0]
    assert q(100) == q(96) == q(127) != q(128)
    # a table with fewer slots than ways has no set
    assert q(31) == q(0)


def test_null_handle_is_rejected():
    lib = pk.load_library()
    assert lib.recmg_embbag_forward(None, None, None, 0, 0, None, None) == bd.RECMG_E_INVALID
    assert lib.recmg_apply_placement(None, None, None, 0, None, None) == bd.RECMG_E_INVALID
    assert lib.recmg_cache_destroy(None) == bd.RECMG_OK


def test_bench_refuses_more_than_one_gpu():
    """bench.py --gpus N > 1 stops before touching a GPU, with a JSON error line and status 2."""
    import json
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=root)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_missing_library_fails_loudly():
    """With no built library the binding raises: there is no other path."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import paper_2511_08568_amd as p\n"
            "try:\n    p.load_library()\nexcept RuntimeError as e:\n    print('raised', e)\n")
    env = dict(os.environ, RECMG_LIBRARY=os.path.join(root, "no_such_librecmg.so"))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120, cwd=root, env=env)
    assert r.returncode == 0 and r.stdout.startswith("raised"), r.stdout + r.stderr


def test_per_table_miss_modes():
    """miss_modes overrides miss_mode per table: one STAGED table is enough for
    pinned host staging; a bad entry is rejected; NULL keeps miss_mode."""
    import ctypes
    base = _cfg(rows=(1000, 2000), dims=(64, 32), dtypes=(0, 0), caps=(100, 100))
    _, host0 = bd.recmg_query_workspace(base)
    assert host0 == 0
    modes = (ctypes.c_int32 * 2)(0, 1)
    base.miss_modes = modes
    _, host1 = bd.recmg_query_workspace(base)
    assert host1 > 0
    bad = (ctypes.c_int32 * 2)(0, 7)
    base.miss_modes = bad
    with pytest.raises(bd.RecmgError) as e:
        bd.recmg_query_workspace(base)
    assert e.value.code == bd.RECMG_E_INVALID and "miss_modes" in pk.recmg_last_error()
