"""recmg_cache_init_static (the entry point for callers that cannot allocate
device memory) against recmg_cache_init on the same calls: every counter and
resident set equal, pooled sums equal bit for bit (the same kernels sum each
bag in a fixed order) and within rtol x L1 mass of the oracle.  Two handles in
a row on the device's static array, the second with a smaller configuration,
so the second starts from what the first left there."""
import ctypes

import numpy as np
import pytest

import tracegen as tg
from _helpers import FWD_KEYS, PLACE_KEYS, check_pooled

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from paper_2511_08568_amd import RecmgError, TieredEmbeddingCache  # noqa: E402
from paper_2511_08568_amd import binding as bd  # noqa: E402


def _caches(w, tabs, nb):
    host = [torch.from_numpy(np.ascontiguousarray(a)).pin_memory() for a in tabs]
    kw = dict(policy=w.policy, eviction_speed=w.eviction_speed, max_bags_per_table=w.bags,
              max_indices=max(w.batch(b)[0].size for b in range(nb)),
              max_prefetch=max(max(w.prefetch_list(b)[0].size for b in range(nb)), 1), ways=w.ways)
    dt = [tb.dtype for tb in w.tables]
    caps = [tb.cap for tb in w.tables]
    return host, TieredEmbeddingCache(host, dt, caps, static_workspace=True, **kw), TieredEmbeddingCache(host, dt, caps, **kw)


def _compare(w, nb, label):
    import oracle
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    f64 = [tg.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
    host, st, ref = _caches(w, tabs, nb)
    assert st.workspace is None  # nothing allocated for the static handle's workspace
    o = oracle.for_workload(w, tabs)
    dev = torch.device("cuda", 0)
    try:
        for b in range(nb):
            P, poff = w.prefetch_list(b)
            bits = w.cache_bits(b - 1) if b > 0 else None
            dP = torch.from_numpy(P).to(dev) if P.size else None
            dpo = torch.from_numpy(poff).to(dev)
            dbits = None if bits is None else torch.from_numpy(bits).to(dev)
            for c in (st, ref):
                c.placement(dP, dpo, dbits)
            assert o.placement(P, poff, bits) == 0
            (ls, _, rs), (lr, _, rr) = st.stats(dump=True), ref.stats(dump=True)
            for t in range(w.num_tables):
                for k in PLACE_KEYS:
                    assert ls[t][k] == lr[t][k], f"{label} placement {b} table {t} {k}"
                assert np.array_equal(rs[t], rr[t]) and np.array_equal(rs[t], o.resident(t)), f"{label} {b} {t}"
            idx, off = w.batch(b)
            di, do = torch.from_numpy(idx).to(dev), torch.from_numpy(off).to(dev)
            out_s = st.forward(di, do, w.bags).cpu().numpy()
            out_r = ref.forward(di, do, w.bags).cpu().numpy()
            _, _, r64 = o.forward(idx, off, w.bags, want64=True)
            (ls, _), (lr, _) = st.stats(), ref.stats()
            for t in range(w.num_tables):
                for k in FWD_KEYS:
                    assert ls[t][k] == lr[t][k] == o.stats(t)[k], f"{label} forward {b} table {t} {k}"
            assert np.array_equal(out_s, out_r), f"{label} batch {b}: pooled sums differ between the entry points"
            check_pooled(w, f64, idx, off, out_s, r64, f"{label} batch {b}")
    finally:
        st.close()
        ref.close()
        o.close()


def test_static_workspace_matches_the_allocating_entry_point():
    # configuration 1 at full size (1 x 100,000 x 64 fp32, cache 10,000), then
    # a smaller one: 2 tables, LRU and 8-way sets, on the array the first left
    w1 = tg.make_config(1)
    _compare(w1, 6, "c1")
    w2 = tg.scaled_config(2, row_scale=0.002, batches=4, bags=64, max_tables=2, ways=8)
    _compare(w2, 4, "c2-small-8way")


def _cfg_for(host, caps):
    T = len(host)
    keep = dict(rows=(ctypes.c_int64 * T)(*[h.shape[0] for h in host]),
                dims=(ctypes.c_int32 * T)(*[h.shape[1] for h in host]),
                dtypes=(ctypes.c_int32 * T)(*([bd.RECMG_F32] * T)),
                ptrs=(ctypes.c_void_p * T)(*[h.data_ptr() for h in host]),
                caps=(ctypes.c_int64 * T)(*caps))
    cfg = bd.recmg_config_t()
    cfg.num_tables, cfg.rows, cfg.dims, cfg.dtypes = T, keep["rows"], keep["dims"], keep["dtypes"]
    cfg.host_tables, cfg.cache_rows = keep["ptrs"], keep["caps"]
    cfg.max_bags_per_table, cfg.max_indices, cfg.max_prefetch = 64, 4096, 4096
    cfg._keep = keep
    return cfg


def test_static_workspace_limits():
    """Over-size configurations get RECMG_E_NOMEM; a second live handle on the
    device gets RECMG_E_STATE until the first is destroyed."""
    lib = bd.load_library()
    small = [torch.zeros((1000, 64), dtype=torch.float32).pin_memory()]
    big = [torch.zeros((200000, 128), dtype=torch.float32).pin_memory()]
    cfg_big = _cfg_for(big, [100000])  # 51 MB of slots alone
    need, _ = bd.recmg_query_workspace(cfg_big)
    assert need > 32 << 20
    h = ctypes.c_void_p(0)
    assert lib.recmg_cache_init_static(ctypes.byref(cfg_big), ctypes.byref(h)) == bd.RECMG_E_NOMEM
    assert not h.value and "static workspace" in bd.recmg_last_error()
    cfg = _cfg_for(small, [100])
    h1 = ctypes.c_void_p(0)
    assert lib.recmg_cache_init_static(ctypes.byref(cfg), ctypes.byref(h1)) == bd.RECMG_OK and h1.value
    h2 = ctypes.c_void_p(0)
    assert lib.recmg_cache_init_static(ctypes.byref(cfg), ctypes.byref(h2)) == bd.RECMG_E_STATE and not h2.value
    assert lib.recmg_cache_destroy(h1) == bd.RECMG_OK
    assert lib.recmg_cache_init_static(ctypes.byref(cfg), ctypes.byref(h2)) == bd.RECMG_OK and h2.value
    assert lib.recmg_cache_destroy(h2) == bd.RECMG_OK
    with pytest.raises(RecmgError):
        bd.recmg_cache_init_static(cfg_big)
