"""HIP path vs the CPU oracle at the full sizes of configurations 2-5, in the
launch configuration bench.py times: placements on a stream of their own,
calls issued back to back with no synchronisation between them.

Checked: every call's counters and every placement's digest (the device stats
log) against the oracle replaying the same calls, the final resident sets row
by row, and the pooled sums of every bag of the first and last batch, summed
on the host in fp64 from the tables (the oracle's definition) and compared
element by element within rtol x the element's L1 mass.  Configurations 4
and 5 run in STAGED mode (their 102 and 61 GB of tables stay pageable).
Configuration 1 at full size is in test_gpu_parity.py."""
import gc
import os
import sys
import time

import numpy as np
import pytest

import tracegen as tg

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

RTOL = {"f32": 1e-5, "f16": 2e-2, "bf16": 2e-2}
TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.uint16}


def _say(msg):
    print(f"[fullsize] {msg}", file=sys.stderr, flush=True)


def _run(cid, nb, miss_mode="zero_copy", ways=0, start=0, warm=0):
    """nb steps of configuration cid on batches start .. start + nb - 1, after
    `warm` warm-up placements (no forward between them) that fill every cache
    with its Cap most popular rows."""
    import oracle
    from paper_2511_08568_amd import TieredEmbeddingCache
    w = tg.make_config(cid)
    w.ways = ways
    dev = torch.device("cuda", 0)
    t0 = time.time()
    pin = miss_mode == "zero_copy"
    host = [torch.empty((tb.rows, tb.dim), dtype=TDT[tb.dtype], pin_memory=pin) for tb in w.tables]
    for t in range(w.num_tables):
        w.table_values(t, out=host[t].numpy())
    _say(f"config {cid}: tables ready in {time.time() - t0:.1f}s")
    batches = [w.batch(start + b) for b in range(nb)]
    pre = [w.prefetch_list(start + b) for b in range(nb)]
    bits = [w.cache_bits(start + b - 1) if b > 0 else None for b in range(nb)]
    warm_lists = [w.warm_list(k, warm) for k in range(warm)]
    _say(f"config {cid}: batches {start}..{start + nb - 1} and {warm} warm-up lists drawn")
    d_warm = [(torch.from_numpy(P).to(dev), torch.from_numpy(po).to(dev)) for P, po in warm_lists]
    d_in = []
    for b in range(nb):
        (idx, off), (P, po) = batches[b], pre[b]
        d_in.append((torch.from_numpy(P).to(dev) if P.size else None, torch.from_numpy(po).to(dev),
                     None if bits[b] is None else torch.from_numpy(bits[b]).to(dev),
                     torch.from_numpy(idx).to(dev), torch.from_numpy(off).to(dev)))
    cache = TieredEmbeddingCache(host, [tb.dtype for tb in w.tables], [tb.cap for tb in w.tables], policy=w.policy,
                                 eviction_speed=w.eviction_speed, miss_mode=miss_mode, max_bags_per_table=w.bags,
                                 max_indices=max(i.size for i, _ in batches),
                                 max_prefetch=max(max(P.size for P, _ in pre + warm_lists), 1), ways=ways,
                                 stats_log_calls=2 * nb + warm)
    outs = [torch.empty(w.bags * sum(tb.dim for tb in w.tables), dtype=torch.float32, device=dev) for _ in range(nb)]
    pstream = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    try:
        for P, po in d_warm:
            cache.placement(P, po, None, stream=pstream)
        for b in range(nb):
            P, po, cb, idx, off = d_in[b]
            cache.placement(P, po, cb, stream=pstream)
            cache.forward(idx, off, w.bags, out=outs[b])
        log = cache.stats_log()
        _, _, res = cache.stats(dump=True)
    finally:
        cache.close()
    del cache, d_in, d_warm
    _say(f"config {cid}: {warm} warm-up placements and {nb} steps on the GPU done")
    host_np = [h.numpy() for h in host]
    nth = max(1, min(16, len(os.sched_getaffinity(0)), w.num_tables))
    o = oracle.for_workload(w, host_np, nthreads=nth)
    evicted = 0
    try:
        for k, (P, po) in enumerate(warm_lists):
            assert o.placement(P, po, None) == 0
            for t in range(w.num_tables):
                st = o.stats(t)
                for key in oracle.PLC_FIELDS + ("digest",):
                    assert log[k][t][key] == st[key], f"config {cid} warm-up placement {k} table {t} {key}"
            _say(f"config {cid}: warm-up placement {k} equal")
        for b in range(nb):
            (idx, off), (P, po) = batches[b], pre[b]
            assert o.placement(P, po, bits[b]) == 0
            for t in range(w.num_tables):
                st = o.stats(t)
                evicted += st["evicted"]
                for k in oracle.PLC_FIELDS + ("digest",):
                    assert log[warm + 2 * b][t][k] == st[k], f"config {cid} placement {start + b} table {t} {k}"
            assert o.forward(idx, off, w.bags)[0] == 0
            for t in range(w.num_tables):
                st = o.stats(t)
                for k in oracle.FWD_FIELDS:
                    assert log[warm + 2 * b + 1][t][k] == st[k], f"config {cid} forward {start + b} table {t} {k}"
            if warm:
                _say(f"config {cid}: batch {start + b} equal")
        for t in range(w.num_tables):
            assert np.array_equal(res[t], o.resident(t)), f"config {cid} table {t}: final resident set"
    finally:
        o.close()
    _say(f"config {cid}: counters and resident sets equal the oracle's ({evicted} evictions)")
    # every bag of the first and last batch, summed in fp64 on the host from
    # the tables (the oracle's definition), table by table
    for b in sorted({0, nb - 1}):
        idx, off = batches[b]
        got = outs[b].cpu().numpy()
        base = 0
        for t, tb in enumerate(w.tables):
            o0 = int(off[t * w.bags])
            seg = off[t * w.bags: (t + 1) * w.bags + 1] - o0
            rows = tg.storage_to_f64(host_np[t][idx[o0:o0 + int(seg[-1])]], tb.dtype)
            ref = np.zeros((w.bags, tb.dim))
            mass = np.zeros((w.bags, tb.dim))
            full = seg[1:] > seg[:-1]  # non-empty bags; each sums up to the next one's start
            if full.any():
                ref[full] = np.add.reduceat(rows, seg[:-1][full], axis=0)
                mass[full] = np.add.reduceat(np.abs(rows), seg[:-1][full], axis=0)
            g = got[base: base + w.bags * tb.dim].reshape(w.bags, tb.dim).astype(np.float64)
            bad = np.abs(g - ref) > RTOL[tb.dtype] * mass
            assert not bad.any(), (f"config {cid} batch {start + b} table {t}: {int(bad.sum())} outputs outside "
                                   f"tolerance, first in bag {int(np.argwhere(bad)[0][0])}")
            base += w.bags * tb.dim
            del rows, ref, mass, g
    _say(f"config {cid}: every pooled sum of the first and last batch within tolerance")
    return evicted


def _release():
    """Give back device memory and pinned host memory that torch keeps cached:
    the box caps pinned memory, and these tests pin tens of GB each."""
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch._C._host_emptyCache()


@pytest.fixture(autouse=True)
def _free_between_tests():
    _release()
    yield
    _release()


def test_config2_fullsize():
    """8 x 1,000,000 x 128 fp32, cache 50,000/table, 2,048 bags: 8 steps."""
    _run(2, 8)


def test_config2_fullsize_32way():
    _run(2, 6, ways=32)


def test_config3_fullsize():
    """26 fp16 tables (1e3..2e7 rows), cache 2%, 4,096 bags: 5 steps."""
    _run(3, 5)


def test_config4_fullsize_staged():
    """4 x 1e8 x 128 bf16 (102 GB, pageable), 20 GB cache, 16,384 bags of 80: 3 steps."""
    _run(4, 3, miss_mode="staged")


def test_config4_fullsize_steady_state():
    """Configuration 4 with its 20 GB cache full: five warm-up placements name
    each table's 19,531,250 most popular rows (78.1M resident keys), then
    batches 46-55 with exact prefetch cross the drift at batch 50 (10% of the
    lookups move to a new hot set).  Every placement evicts and ranks over the
    full caches; every call's counters and digests, the final resident sets
    and sampled pooled sums are checked against the oracle."""
    evicted = _run(4, 10, miss_mode="staged", start=46, warm=5)
    assert evicted > 0


def test_config5_fullsize_staged():
    """64 x 2,000,000 fp32 (dims 32..256, 61 GB, pageable), cache 10%, 8,192 bags: 4 steps."""
    _run(5, 4, miss_mode="staged")
