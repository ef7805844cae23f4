"""Error paths of the C ABI on the GPU.  Every condition is either rejected on
the host or detected by a kernel's own range checks before any access, so no
kernel reads or writes outside its buffers."""
import numpy as np
import pytest

import tracegen as tg
from _helpers import GpuRunner

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

from paper_2511_08568_amd import RecmgError  # noqa: E402
from paper_2511_08568_amd import binding as bd  # noqa: E402


def _workload():
    return tg.scaled_config(1, row_scale=0.01, batches=3, bags=32)


def _runner(validate=False):
    w = _workload()
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    return w, GpuRunner(w, tabs, validate=validate)


def test_validate_mode_rejects_bad_rows_and_keeps_state():
    w, g = _runner(validate=True)
    try:
        P, poff = w.prefetch_list(0)
        g.placement(P, poff)
        before, _, res_before = g.cache.stats(dump=True)
        idx, off = w.batch(0)
        bad = idx.copy()
        bad[3] = w.tables[0].rows  # one past the end
        with pytest.raises(RecmgError) as e:
            g.forward(bad, off)
        assert e.value.code == bd.RECMG_E_RANGE
        badP = P.copy()
        badP[0] = -1
        with pytest.raises(RecmgError) as e:
            g.placement(badP, poff)
        assert e.value.code == bd.RECMG_E_RANGE
        after, _, res_after = g.cache.stats(dump=True)
        assert before == after and all(np.array_equal(a, b) for a, b in zip(res_before, res_after))
        g.forward(idx, off)  # a good call still works
    finally:
        g.close()


def test_device_detects_bad_row_and_latches():
    w, g = _runner()
    try:
        P, poff = w.prefetch_list(0)
        g.placement(P, poff)
        idx, off = w.batch(0)
        bad = idx.copy()
        bad[-1] = w.tables[0].rows + 1000
        g.forward(bad, off)  # asynchronous: the device latches the error
        _, _, code = g.cache.stats(strict=False)
        assert code == bd.RECMG_E_RANGE
        g.forward(idx, off)  # later calls are no-ops on the device
        _, _, code = g.cache.stats(strict=False)
        assert code == bd.RECMG_E_RANGE
    finally:
        g.close()


def test_device_detects_malformed_offsets():
    w, g = _runner()
    try:
        idx, off = w.batch(0)
        bad = off.copy()
        bad[6] = bad[5] - 1  # offsets decrease
        assert bad[5] > 0
        g.forward(idx, bad)
        _, _, code = g.cache.stats(strict=False)
        assert code == bd.RECMG_E_RANGE
    finally:
        g.close()


def test_host_rejects_oversize_and_null_arguments():
    w, g = _runner()
    try:
        idx, off = w.batch(0)
        h = g.cache.handle
        dev_idx, dev_off = g.to_dev(idx), g.to_dev(off)
        out = torch.empty(w.bags * w.tables[0].dim, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        # more indices than max_indices
        assert bd.recmg_embbag_forward(h, dev_idx.data_ptr(), dev_off.data_ptr(), 10**9, w.bags, out.data_ptr(),
                                       s) == bd.RECMG_E_INVALID
        # more bags than max_bags_per_table
        assert bd.recmg_embbag_forward(h, dev_idx.data_ptr(), dev_off.data_ptr(), idx.size, w.bags + 1,
                                       out.data_ptr(), s) == bd.RECMG_E_INVALID
        # null offsets / prefetch offsets
        assert bd.recmg_embbag_forward(h, dev_idx.data_ptr(), 0, idx.size, w.bags, out.data_ptr(),
                                       s) == bd.RECMG_E_INVALID
        assert bd.recmg_apply_placement(h, 0, 0, 0, 0, s) == bd.RECMG_E_INVALID
        assert bd.recmg_apply_placement(h, 0, dev_off.data_ptr(), 10**9, 0, s) == bd.RECMG_E_INVALID
        assert bd.recmg_last_error()
        # nothing was launched: the cache still works and is empty
        last, _ = g.cache.stats()
        assert last[0]["resident"] == 0
    finally:
        g.close()


def test_empty_batches_and_empty_prefetch():
    w = tg.scaled_config(1, row_scale=0.01, batches=2, bags=16)
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    g = GpuRunner(w, tabs, max_indices=64, max_prefetch=64)
    try:
        g.placement(np.zeros(0, np.int32), np.zeros(2, np.int64))
        off = np.zeros(w.bags + 1, np.int64)  # every bag empty
        out = g.cache.forward(g.to_dev(np.zeros(1, np.int32))[:0], g.to_dev(off), w.bags).cpu().numpy()
        assert out.shape == (w.bags * w.tables[0].dim,) and not out.any()
        last, _ = g.cache.stats()
        assert last[0]["lookups"] == 0 and last[0]["unique"] == 0 and last[0]["misses"] == 0
        # zero bags
        out0 = g.cache.forward(g.to_dev(np.zeros(1, np.int32))[:0], g.to_dev(np.zeros(1, np.int64)), 0)
        assert out0.numel() == 0
        g.placement(np.zeros(0, np.int32), np.zeros(2, np.int64))
        last, _ = g.cache.stats()
        assert last[0]["resident"] == 0
    finally:
        g.close()


def test_destroy_accepts_null_and_close_is_idempotent():
    """recmg_cache_destroy(NULL) is a no-op; the binding's close() releases the
    handle once and forgets it, so a second close() calls nothing.  (A handle
    pointer is dangling after destroy, so no call is made with it.)"""
    w, g = _runner()
    g.close()
    assert g.cache.handle == 0
    g.close()
    assert bd.recmg_cache_destroy(0) == bd.RECMG_OK


def test_init_reports_nomem_through_the_c_abi():
    """recmg_cache_init itself returns RECMG_E_NOMEM for a device workspace
    shorter than recmg_query_workspace asks for (and for none at all), and
    sets no handle."""
    import ctypes
    w = _workload()
    tab = torch.from_numpy(w.table_values(0)).pin_memory()
    rows = (ctypes.c_int64 * 1)(tab.shape[0])
    dims = (ctypes.c_int32 * 1)(tab.shape[1])
    dts = (ctypes.c_int32 * 1)(bd.RECMG_F32)
    caps = (ctypes.c_int64 * 1)(10)
    ptrs = (ctypes.c_void_p * 1)(tab.data_ptr())
    cfg = bd.recmg_config_t()
    cfg.num_tables, cfg.rows, cfg.dims, cfg.dtypes, cfg.host_tables, cfg.cache_rows = 1, rows, dims, dts, ptrs, caps
    cfg.max_bags_per_table, cfg.max_indices, cfg.max_prefetch = 8, 64, 64
    need, _ = bd.recmg_query_workspace(cfg)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    lib = bd.load_library()
    for size, ptr in ((need - 256, ws.data_ptr()), (need, 0)):
        cfg.device_workspace, cfg.device_workspace_bytes = ptr, size
        h = ctypes.c_void_p(0)
        assert lib.recmg_cache_init(ctypes.byref(cfg), ctypes.byref(h)) == bd.RECMG_E_NOMEM
        assert not h.value and "workspace" in bd.recmg_last_error()
    # the full size is accepted
    cfg.device_workspace, cfg.device_workspace_bytes = ws.data_ptr(), need
    h = ctypes.c_void_p(0)
    assert lib.recmg_cache_init(ctypes.byref(cfg), ctypes.byref(h)) == bd.RECMG_OK and h.value
    assert lib.recmg_cache_destroy(h) == bd.RECMG_OK


def test_init_rejects_small_workspace_and_pageable_tables():
    from paper_2511_08568_amd import TieredEmbeddingCache
    w = _workload()
    tab = torch.from_numpy(w.table_values(0))
    with pytest.raises(ValueError):
        TieredEmbeddingCache([tab], ["f32"], [10], max_bags_per_table=8, max_indices=64, max_prefetch=64)
    pinned = tab.pin_memory()
    with pytest.raises(ValueError):
        TieredEmbeddingCache([pinned], ["f32"], [10], max_bags_per_table=8, max_indices=64, max_prefetch=64,
                             workspace=torch.empty(16, dtype=torch.uint8, device="cuda"))
