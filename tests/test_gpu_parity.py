"""HIP path vs the CPU oracle, through the C ABI: counters and resident sets
bit-exact, pooled outputs within rtol * L1 mass (1e-5 fp32, 2e-2 fp16/bf16)."""
import numpy as np
import pytest

import tracegen as tg
from _helpers import GpuRunner, check_pooled, compare_runs, golden_table, load_golden
from oracle_pins import GOLDEN_FILES, run_oracle

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _parity(w, nbatches=None, miss_mode="zero_copy", label="", pin=True):
    """The HIP path against the oracle on w's batches (miss_mode: one mode or one per table)."""
    nb = nbatches or w.batches
    tabs, ora = run_oracle(w, nbatches=nb)
    g = GpuRunner(w, tabs, miss_mode=miss_mode, nbatches=nb, pin=pin)
    try:
        gpu = g.run(nb)
    finally:
        g.close()
    return compare_runs(w, tabs, ora, gpu, label=label or w.name)


@pytest.mark.parametrize("name", GOLDEN_FILES)
def test_hand_examples(name):
    gd = load_golden(name)
    tab = golden_table(gd)
    w = tg.Workload(0, name, [tg.Table(gd["rows"], gd["dim"], "f32", gd["cap"], 1.0, ("fixed", 1))],
                    batches=len(gd["steps"]), bags=1, policy=gd["policy"], eviction_speed=gd["eviction_speed"],
                    ways=gd.get("ways", 0))
    import torch as th
    from paper_2511_08568_amd import TieredEmbeddingCache
    dev = th.device("cuda", 0)
    cache = TieredEmbeddingCache([th.from_numpy(tab).pin_memory()], ["f32"], [gd["cap"]], policy=gd["policy"],
                                 eviction_speed=gd["eviction_speed"], max_bags_per_table=4, max_indices=16,
                                 max_prefetch=16, ways=w.ways)
    for b, step in enumerate(gd["steps"]):
        P = np.array(step["prefetch"], np.int32)
        bits = None if step["bits"] is None else th.tensor(step["bits"], dtype=th.uint8, device=dev)
        cache.placement(th.from_numpy(P).to(dev) if P.size else None, th.tensor([0, P.size], device=dev), bits)
        last, _, res = cache.stats(dump=True)
        for k, v in step["expect_placement"].items():
            assert last[0][k] == v, (name, b, k)
        assert res[0].tolist() == step["resident"], (name, b)
        off = np.array(step["offsets"], np.int64)
        out = cache.forward(th.tensor(step["indices"], dtype=th.int32, device=dev), th.from_numpy(off).to(dev),
                            off.size - 1)
        last, _ = cache.stats()
        for k, v in step["expect_forward"].items():
            assert last[0][k] == v, (name, b, k)
        assert out.cpu().numpy().tolist() == np.array(step["out"], np.float32).reshape(-1).tolist()
    cache.close()


@pytest.mark.parametrize("seed", range(24))
def test_tiny_random(seed):
    w = tg.random_tiny(seed, max_rows=40, max_cap=12, max_dim=9, batches=6, bags=5)
    _parity(w, label=f"tiny{seed}")


@pytest.mark.parametrize("seed", range(6))
def test_lru_ring_long_runs(seed):
    """LRU_BATCH fully associative tables keep their residents in a key-ordered
    ring: 60 placements on caches of at most 300 rows with prefetch lists of
    every kind, so that the ring compacts (its buffers hold Cap plus three
    placements' worth of appends) and some placements drop more keys than the
    ring holds live (the threshold then falls among this placement's own
    keys); every placement's counters, digest and resident set against the
    oracle."""
    w = tg.random_tiny(800 + seed, max_rows=3000, max_cap=300, max_dim=17, batches=60, bags=40,
                       integer_values=False, policy="lru")
    _parity(w, label=f"ring{seed}")


@pytest.mark.parametrize("seed", range(6))
def test_small_random_real_values(seed):
    w = tg.random_tiny(100 + seed, max_rows=3000, max_cap=600, max_dim=70, batches=5, bags=40,
                       integer_values=False)
    _parity(w, label=f"small{seed}")


def test_config1_full():
    """Config 1 at full size (1 x 100,000 x 64 fp32, cache 10,000), first 40 batches."""
    _parity(tg.make_config(1), nbatches=40)


@pytest.mark.parametrize("cid,scale,bags,tables", [(2, 0.02, 256, 3), (3, 0.01, 256, 6), (4, 0.0005, 512, 2),
                                                   (5, 0.01, 256, 8)])
def test_configs_scaled(cid, scale, bags, tables):
    """Configs 2-5 with rows and caches scaled down (same dims, dtypes, policies,
    pooling laws, Zipf exponents and prefetch recipes), several tiles of rows
    per table and ragged bags."""
    w = tg.scaled_config(cid, row_scale=scale, batches=6, bags=bags, max_tables=tables)
    _parity(w, label=f"c{cid}-scaled")


@pytest.mark.parametrize("ways,policy", [(0, "priority"), (0, "lru"), (16, "priority")])
def test_dedup_bitmap_slices(ways, policy):
    """Row counts on both sides of the dedup's limits: a bitmap of exactly one
    LDS slice (2^20 rows), one row more (a second, nearly empty slice), exactly
    the most slices marked in LDS (2^25 rows) and one row more (marked with
    device atomics, beside the others in the same call), and a small table."""
    rows = [1 << 20, (1 << 20) + 1, 1 << 25, (1 << 25) + 1, 3000]
    tabs = [tg.Table(n, 4, "f32", 1500 if ways == 0 else 1024, a, ("poisson", 20.0, 1, 60))
            for n, a in zip(rows, (0.9, 1.1, 1.0, 1.2, 1.05))]
    w = tg.Workload(0, f"dedup-slices-w{ways}-{policy}", tabs, batches=6, bags=512, policy=policy,
                    prefetch=("mix", 0.7), ways=ways)
    _parity(w)


# Row sizes that pick each pooled-kernel shape: 64 and 128 bytes (4 or 2 rows
# per load instruction), 256 / 512 / 1024 bytes (one row per instruction, 4, 8
# or 16 bytes per lane), 2048 bytes (two chunks per row), and sizes the
# wave-per-bag kernel does not take (the group-per-bag kernel, vector and
# scalar forms).
POOL_DIMS = {"f32": [16, 32, 64, 128, 256, 512, 24, 7],
             "f16": [32, 64, 128, 256, 512, 1024, 40, 5],
             "bf16": [32, 64, 128, 256, 512, 1024, 40, 5]}


def _kinds_workload(dtypes, seed, policy):
    """Tables of every pooled-kernel shape (interleaved dtypes when several),
    ragged bags: empty, single-row, shorter and longer than one block of
    loads, and long geometric tails."""
    g = np.random.default_rng(seed)
    tabs = []
    pools = [("poisson", 6.0, 0, 200), ("geometric", 45.0), ("poisson", 70.0, 1, 200), ("onehot",)]
    for k in range(max(len(POOL_DIMS[d]) for d in dtypes)):
        for d in dtypes:
            dims = POOL_DIMS[d]
            if k < len(dims):
                rows = int(g.integers(500, 4000))
                tabs.append(tg.Table(rows, dims[k], d, int(rows * g.uniform(0.02, 0.3)),
                                     float(g.uniform(0.8, 1.3)), pools[(k + len(tabs)) % len(pools)]))
    return tg.Workload(900 + seed, f"kinds{seed}", tabs, batches=4, bags=37, policy=policy,
                       prefetch=("mix", 0.7))


@pytest.mark.parametrize("dtypes,seed,policy", [(("f32",), 1, "lru"), (("f16",), 2, "priority"),
                                                (("bf16",), 3, "lru"), (("bf16", "f32", "f16"), 4, "priority")])
def test_pool_kernel_shapes(dtypes, seed, policy):
    _parity(_kinds_workload(dtypes, seed, policy), label=f"kinds-{'-'.join(dtypes)}")


@pytest.mark.parametrize("cid,scale,tables", [(3, 0.01, 6), (5, 0.005, 8)])
def test_optgen_caching_bits(cid, scale, tables):
    """PRIORITY placement fed OPTgen's Belady-optimal labels (the caching
    model's ground truth, Sec. VI-A) instead of the noisy lookahead bits."""
    w = tg.scaled_config(cid, row_scale=scale, batches=6, bags=256, max_tables=tables)
    w.bits = ("optgen", 0.8, w.batches)
    _parity(w, label=f"c{cid}-optgen")


@pytest.mark.parametrize("prefetch", ["exact", "none"])
def test_config4_scaled_steady_state_across_drift(prefetch):
    """Scaled configuration 4 (2 tables of 50,000 rows, cache 9,766 each)
    started full by three warm-up placements, then batches 46-55, across the
    drift at batch 50: every call against the oracle, with evictions in every
    placement once the cache is full."""
    import oracle
    w = tg.scaled_config(4, row_scale=0.0005, batches=200, bags=512, max_tables=2, prefetch=(prefetch,))
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    f64 = [tg.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
    o = oracle.for_workload(w, tabs)
    warm = [w.warm_list(k, 3) for k in range(3)]
    maxp = max(max(P.size for P, _ in warm), max(w.prefetch_list(b)[0].size for b in range(46, 56)), 1)
    g = GpuRunner(w, tabs, max_indices=max(w.batch(b)[0].size for b in range(46, 56)), max_prefetch=maxp)
    evicted = 0
    try:
        for P, po in warm:
            g.placement(P, po)
            assert o.placement(P, po) == 0
        last, _ = g.cache.stats()
        assert all(last[t]["resident"] == w.tables[t].cap for t in range(w.num_tables))
        for b in range(46, 56):
            P, po = w.prefetch_list(b)
            g.placement(P, po)
            assert o.placement(P, po) == 0
            last, _, res = g.cache.stats(dump=True)
            for t in range(w.num_tables):
                for k in ("evicted", "admitted_miss", "prefetch_fill", "prefetch_resident", "prefetch_dropped",
                          "miss_dropped", "resident", "prefetch_distinct", "digest"):
                    assert last[t][k] == o.stats(t)[k], f"batch {b} table {t} placement {k}"
                assert np.array_equal(res[t], o.resident(t))
                evicted += last[t]["evicted"]
            idx, off = w.batch(b)
            out = g.forward(idx, off)
            st, _, r64 = o.forward(idx, off, w.bags, want64=True)
            last, _ = g.cache.stats()
            for t in range(w.num_tables):
                for k in ("lookups", "unique", "hits", "hits_prefetch", "misses", "prefetch_covered"):
                    assert last[t][k] == o.stats(t)[k], f"batch {b} table {t} forward {k}"
            check_pooled(w, f64, idx, off, out, r64, f"batch {b}")
    finally:
        g.close()
        o.close()
    assert evicted > 0


def test_config4_no_prefetch_scaled():
    w = tg.scaled_config(4, row_scale=0.0005, batches=6, bags=512, max_tables=2, prefetch=("none",))
    _parity(w, label="c4-noprefetch")


def test_staged_matches_oracle():
    w = tg.scaled_config(3, row_scale=0.01, batches=5, bags=256, max_tables=5)
    _parity(w, miss_mode="staged", label="c3-staged")


@pytest.mark.parametrize("cid,scale,tables", [(3, 0.01, 5), (4, 0.0005, 2), (5, 0.005, 6)])
def test_staged_with_unpinned_tables(cid, scale, tables):
    """STAGED mode never reads host tables from the GPU (misses and prefetch
    fills are gathered on the host), so the tables may be ordinary memory."""
    w = tg.scaled_config(cid, row_scale=scale, batches=5, bags=256, max_tables=tables)
    _parity(w, miss_mode="staged", label=f"c{cid}-staged-unpinned", pin=False)


@pytest.mark.parametrize("cid,scale,tables,ways", [(4, 0.0005, 4, 0), (3, 0.01, 5, 0), (5, 0.005, 6, 32)])
def test_mixed_miss_modes(cid, scale, tables, ways):
    """Per-table miss modes: the first half of the tables pinned and read
    zero-copy, the rest ordinary memory gathered on the host, in one handle
    (the configuration-4 setup where only some tables fit the pinned-memory
    limit), against the oracle."""
    w = tg.scaled_config(cid, row_scale=scale, batches=5, bags=256, max_tables=tables, ways=ways)
    modes = ["zero_copy" if t < tables // 2 else "staged" for t in range(tables)]
    _parity(w, miss_mode=modes, label=f"c{cid}-mixed", pin=False)


@pytest.mark.parametrize("overlap,sync,mode", [(True, True, "zero_copy"), (True, False, "zero_copy"),
                                               (False, False, "zero_copy"), (True, False, "staged")])
def test_two_placements_in_a_row(overlap, sync, mode):
    """Two placements in a row (no forward between), each on a stream other
    than the last call's, then a forward on a third stream.  The second
    placement frees slots the first one's fill may still be writing; its fill
    must run after that one.  overlap=False: no copy stream, so every fill runs
    on its own placement's stream.  sync=False: no synchronisation between
    calls (the resident sets are then checked at the end of each batch)."""
    import torch as th
    w = tg.scaled_config(2, row_scale=0.01, batches=4, bags=128, max_tables=2)
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    f64 = [tg.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
    import oracle
    o = oracle.for_workload(w, tabs)
    g = GpuRunner(w, tabs, overlap=overlap, miss_mode=mode)
    streams = [th.cuda.Stream(), th.cuda.Stream(), th.cuda.Stream()]
    try:
        for b in range(w.batches):
            for rep in range(2):
                P, poff = w.prefetch_list(b + rep)
                s = streams[rep]
                with th.cuda.stream(s):
                    g.cache.placement(g.to_dev(P) if P.size else None, g.to_dev(poff), None, stream=s)
                assert o.placement(P, poff) == 0
                if sync:
                    last, _, res = g.cache.stats(dump=True)
                    for t in range(w.num_tables):
                        assert res[t].tolist() == o.resident(t).tolist()
                        assert last[t]["digest"] == o.stats(t)["digest"]
            idx, off = w.batch(b)
            s = streams[2]
            with th.cuda.stream(s):
                out = g.cache.forward(g.to_dev(idx), g.to_dev(off), w.bags, stream=s)
            st, _, ref64 = o.forward(idx, off, w.bags, want64=True)
            assert st == 0
            _, _, res = g.cache.stats(dump=True)  # synchronises every stream the calls used
            for t in range(w.num_tables):
                assert res[t].tolist() == o.resident(t).tolist()
            check_pooled(w, f64, idx, off, out.cpu().numpy(), ref64, f"batch {b}")
    finally:
        g.close()
        o.close()


def test_cap_zero_and_full_give_identical_outputs():
    """Metamorphic: the tier that serves a row must not change the pooled sum."""
    base = tg.scaled_config(2, row_scale=0.005, batches=3, bags=128, max_tables=2)
    outs = []
    for cap in ("zero", "full"):
        w = tg.scaled_config(2, row_scale=0.005, batches=3, bags=128, max_tables=2)
        for tb in w.tables:
            tb.cap = 0 if cap == "zero" else tb.rows
        tabs = [w.table_values(t) for t in range(w.num_tables)]
        g = GpuRunner(w, tabs)
        recs = g.run(dump=False)
        g.close()
        outs.append([r["out"] for r in recs])
        if cap == "zero":
            assert all(r["fwd"][t]["hits"] == 0 for r in recs for t in range(w.num_tables))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
    del base


@pytest.mark.parametrize("ways", [0, 32])
def test_zero_copy_staged_and_mixed_bitwise_equal(ways):
    """The miss path changes where rows come from, never a result: zero-copy,
    STAGED and per-table mixes of the two give bit-identical outputs, counters
    and resident sets."""
    runs = []
    for mode in ("zero_copy", "staged", ["zero_copy", "staged", "staged", "zero_copy"],
                 ["staged", "zero_copy", "zero_copy", "staged"]):
        w = tg.scaled_config(5, row_scale=0.005, batches=4, bags=128, max_tables=4, ways=ways)
        tabs = [w.table_values(t) for t in range(w.num_tables)]
        g = GpuRunner(w, tabs, miss_mode=mode)
        runs.append(g.run())
        g.close()
    for other in runs[1:]:
        for a, b in zip(runs[0], other):
            assert np.array_equal(a["out"], b["out"])
            assert a["fwd"] == b["fwd"] and a["place"] == b["place"]
            assert all(np.array_equal(x, y) for x, y in zip(a["resident"], b["resident"]))


def test_run_twice_is_deterministic():
    res = []
    for _ in range(2):
        w = tg.scaled_config(3, row_scale=0.005, batches=4, bags=256, max_tables=4)
        tabs = [w.table_values(t) for t in range(w.num_tables)]
        g = GpuRunner(w, tabs)
        res.append(g.run())
        g.close()
    for a, b in zip(*res):
        assert np.array_equal(a["out"], b["out"]) and a["fwd"] == b["fwd"] and a["place"] == b["place"]


# ----------------------------------------------------------------------------- set-associative

@pytest.mark.parametrize("seed", range(16))
def test_sa_tiny_random(seed):
    """W-way sets (W = 1..5) on tiny tables: few sets, many evictions per set."""
    w = tg.random_tiny(seed, max_rows=40, max_cap=12, max_dim=9, batches=6, bags=5)
    w.ways = 1 + seed % 5
    _parity(w, label=f"sa-tiny{seed}-w{w.ways}")


@pytest.mark.parametrize("seed,ways", [(0, 2), (1, 4), (2, 8), (3, 3)])
def test_sa_crowded_sets(seed, ways):
    """Hundreds of events per set (more than one wave's worth of misses and of
    prefetch rows), sets that never fill, and tables with no set at all
    (Cap < W) next to set-associative ones."""
    w = tg.random_tiny(200 + seed, max_rows=3000, max_cap=40, max_dim=33, batches=5, bags=60,
                       integer_values=False)
    w.ways = ways
    w.tables[0].cap = ways - 1  # no set: nothing is cached
    _parity(w, label=f"sa-crowded{seed}-w{ways}")


@pytest.mark.parametrize("cid,scale,bags,tables,ways", [(2, 0.02, 256, 3, 32), (3, 0.01, 256, 6, 32),
                                                        (5, 0.01, 256, 8, 32), (4, 0.0005, 512, 2, 32),
                                                        (3, 0.01, 256, 4, 4), (2, 0.02, 256, 2, 64),
                                                        (3, 0.01, 256, 4, 48), (2, 0.02, 256, 2, 17)])
def test_sa_configs_scaled(cid, scale, bags, tables, ways):
    """The scaled configurations with W-way set-associative caches (32 ways:
    the production default the paper compares against)."""
    w = tg.scaled_config(cid, row_scale=scale, batches=6, bags=bags, max_tables=tables, ways=ways)
    _parity(w, label=f"c{cid}-sa{ways}")


def test_sa_staged():
    w = tg.scaled_config(3, row_scale=0.01, batches=5, bags=256, max_tables=5, ways=32)
    _parity(w, miss_mode="staged", label="c3-sa32-staged")


def test_sa_config1_full():
    """Configuration 1 at full size with a 32-way cache (10,000 slots: 312 sets
    of 32, 16 slots unused), first 30 batches."""
    w = tg.make_config(1)
    w.ways = 32
    _parity(w, nbatches=30, label="c1-sa32")


@pytest.mark.parametrize("fill", [0xFF, 0x5A])
def test_workspace_contents_do_not_matter(fill):
    """Regression: init must clear every workspace field a first placement
    reads (a placement before any forward once indexed its fill list from an
    uninitialised field)."""
    import torch as th
    from paper_2511_08568_amd import TieredEmbeddingCache
    w = tg.random_tiny(17, max_rows=40, max_cap=12, max_dim=9, batches=6, bags=5)
    tabs, ora = run_oracle(w)
    probe = GpuRunner(w, tabs)
    nbytes = probe.cache.workspace_bytes
    probe.close()
    ws = th.full((nbytes,), fill, dtype=th.uint8, device="cuda")
    g = GpuRunner.__new__(GpuRunner)
    g.torch, g.w, g.dev, g.pstream = th, w, th.device("cuda", 0), None
    g.host = [th.from_numpy(np.ascontiguousarray(a)).pin_memory() for a in tabs]
    g.cache = TieredEmbeddingCache(g.host, [tb.dtype for tb in w.tables], [tb.cap for tb in w.tables],
                                   policy=w.policy, eviction_speed=w.eviction_speed,
                                   max_bags_per_table=w.bags,
                                   max_indices=max(w.batch(b)[0].size for b in range(w.batches)),
                                   max_prefetch=max(max(w.prefetch_list(b)[0].size for b in range(w.batches)), 1),
                                   workspace=ws)
    try:
        gpu = g.run()
    finally:
        g.close()
    compare_runs(w, tabs, ora, gpu, label=f"garbage-workspace-{fill:#x}")


# ----------------------------------------------------------------------------- pipelined placement

def _device_inputs(w, nb, dev):
    import torch as th
    ins = []
    for b in range(nb):
        P, poff = w.prefetch_list(b)
        bits = w.cache_bits(b - 1) if b > 0 else None
        idx, off = w.batch(b)
        ins.append(dict(P=th.from_numpy(P).to(dev) if P.size else None, poff=th.from_numpy(poff).to(dev),
                        bits=None if bits is None else th.from_numpy(bits).to(dev),
                        idx=th.from_numpy(idx).to(dev), off=th.from_numpy(off).to(dev)))
    th.cuda.synchronize()
    return ins


@pytest.mark.parametrize("cid,scale,tables,ways", [(2, 0.02, 3, 0), (3, 0.01, 6, 0), (5, 0.01, 6, 32),
                                                   (4, 0.0005, 2, 0)])
def test_pipelined_placement_matches_oracle(cid, scale, tables, ways):
    """Placements on a stream of their own, all calls issued back to back with
    no synchronisation in between: placement b+1 runs while forward b still
    waits for its fill or pools, and the fill of b+1 while forward b+1
    deduplicates.  Totals of every counter, the final resident set and digest,
    and every batch's pooled sums must equal the oracle's."""
    import torch as th
    w = tg.scaled_config(cid, row_scale=scale, batches=8, bags=256, max_tables=tables, ways=ways)
    nb = w.batches
    tabs, ora = run_oracle(w, nbatches=nb)
    g = GpuRunner(w, tabs, nbatches=nb, pipeline=True, stats_log_calls=2 * nb)
    try:
        ins = _device_inputs(w, nb, g.dev)
        outs = [th.empty(w.bags * sum(tb.dim for tb in w.tables), dtype=th.float32, device=g.dev) for _ in range(nb)]
        for b in range(nb):
            x = ins[b]
            g.cache.placement(x["P"], x["poff"], x["bits"], stream=g.pstream)
            g.cache.forward(x["idx"], x["off"], w.bags, out=outs[b])
        last, tot, res = g.cache.stats(dump=True)
        log = g.cache.stats_log()
    finally:
        g.close()
    from _helpers import FWD_KEYS, PLACE_KEYS
    # every call's own counters, from the device log
    assert len(log) == 2 * nb
    for b in range(nb):
        for t in range(w.num_tables):
            for k in PLACE_KEYS:
                assert log[2 * b][t][k] == ora[b]["place"][t][k], f"placement {b} table {t} {k}"
            for k in FWD_KEYS:
                assert log[2 * b][t][k] == 0 and log[2 * b + 1][t][k] == ora[b]["fwd"][t][k], f"forward {b} {t} {k}"
            assert all(log[2 * b + 1][t][k] == 0 for k in PLACE_KEYS)
    import tracegen
    f64 = [tracegen.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
    for t in range(w.num_tables):
        for k in PLACE_KEYS:
            if k == "digest":
                continue
            assert tot[t][k] == sum(r["place"][t][k] for r in ora), f"table {t} total {k}"
        for k in FWD_KEYS:
            assert tot[t][k] == sum(r["fwd"][t][k] for r in ora), f"table {t} total {k}"
        assert np.array_equal(res[t], ora[-1]["resident"][t]), f"table {t}: final resident set"
        assert last[t]["digest"] == ora[-1]["place"][t]["digest"]
    for b in range(nb):
        check_pooled(w, f64, ora[b]["idx"], ora[b]["off"], outs[b].cpu().numpy(), ora[b]["out64"], f"batch {b}")


@pytest.mark.parametrize("pipeline", [False, True])
@pytest.mark.parametrize("ways,policy", [(0, "priority"), (16, "priority"), (0, "lfu"), (16, "lfu"), (0, "lru"),
                                         (16, "lru")])
def test_skipped_placements(pipeline, ways, policy):
    """Placements the caller skips (the models were late, Sec. VI-C): the
    next placement sees only the most recent forward's rows and misses, and
    the batches in between run on the cache as it stands (and do not count
    for LFU)."""
    import oracle
    w = tg.scaled_config(3, row_scale=0.01, batches=9, bags=256, max_tables=5, ways=ways, policy=policy)
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    f64 = [tg.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
    o = oracle.for_workload(w, tabs)
    g = GpuRunner(w, tabs, pipeline=pipeline)
    try:
        for b in range(w.batches):
            if b % 3 != 2:
                P, poff = w.prefetch_list(b)
                bits = w.cache_bits(b - 1) if b > 0 else None
                g.placement(P, poff, bits)
                assert o.placement(P, poff, bits) == 0
                last, _, res = g.cache.stats(dump=True)
                for t in range(w.num_tables):
                    ref = o.stats(t)
                    for k in PLACE_KEYS_ALL:
                        assert last[t][k] == ref[k], f"batch {b} table {t} placement {k}"
                    assert np.array_equal(res[t], o.resident(t))
            idx, off = w.batch(b)
            out = g.forward(idx, off)
            st, _, ref64 = o.forward(idx, off, w.bags, want64=True)
            assert st == 0
            last, _ = g.cache.stats()
            for t in range(w.num_tables):
                ref = o.stats(t)
                for k in ("lookups", "unique", "hits", "hits_prefetch", "misses", "prefetch_covered"):
                    assert last[t][k] == ref[k], f"batch {b} table {t} forward {k}"
            check_pooled(w, f64, idx, off, out, ref64, f"batch {b}")
    finally:
        g.close()
        o.close()


PLACE_KEYS_ALL = ("evicted", "admitted_miss", "prefetch_fill", "prefetch_resident", "prefetch_dropped",
                  "miss_dropped", "resident", "prefetch_distinct", "digest")


def test_stats_log_window():
    """The log keeps the latest stats_log_calls calls; older ones are refused."""
    from paper_2511_08568_amd import RecmgError
    w = tg.scaled_config(1, row_scale=0.05, batches=5, bags=64)
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    import oracle
    o = oracle.for_workload(w, tabs)
    g = GpuRunner(w, tabs, stats_log_calls=3)
    try:
        recs = []
        for b in range(w.batches):
            P, poff = w.prefetch_list(b)
            g.placement(P, poff)
            assert o.placement(P, poff) == 0
            recs.append([o.stats(t) for t in range(w.num_tables)])
            idx, off = w.batch(b)
            g.forward(idx, off)
            assert o.forward(idx, off, w.bags)[0] == 0
            recs.append([o.stats(t) for t in range(w.num_tables)])
        log = g.cache.stats_log()
        assert len(log) == 3  # calls 7, 8, 9
        assert log[0][0]["hits"] == recs[7][0]["hits"]      # call 7 = forward 3
        assert log[1][0]["digest"] == recs[8][0]["digest"]  # call 8 = placement 4
        assert log[1][0]["resident"] == recs[8][0]["resident"]
        assert log[2][0]["hits"] == recs[9][0]["hits"]      # call 9 = forward 4
        with pytest.raises(RecmgError):
            g.cache.stats_log(first_call=0, n_calls=4)
        with pytest.raises(RecmgError):
            g.cache.stats_log(first_call=8, n_calls=3)  # call 10 not made yet
    finally:
        g.close()
        o.close()


# ----------------------------------------------------------------------------- LFU

@pytest.mark.parametrize("seed", range(8))
def test_lfu_tiny_random(seed):
    w = tg.random_tiny(300 + seed, max_rows=40, max_cap=12, max_dim=9, batches=6, bags=5, policy="lfu")
    w.ways = (0, 0, 1, 2, 3, 4, 0, 8)[seed]
    _parity(w, label=f"lfu-tiny{seed}-w{w.ways}")


@pytest.mark.parametrize("cid,scale,tables,ways", [(2, 0.02, 3, 0), (3, 0.01, 6, 0), (3, 0.01, 6, 32),
                                                   (5, 0.01, 6, 32)])
def test_lfu_configs_scaled(cid, scale, tables, ways):
    """LFU_BATCH (the LFU baseline) on the scaled configurations, fully
    associative and 32-way."""
    w = tg.scaled_config(cid, row_scale=scale, batches=6, bags=256, max_tables=tables, ways=ways, policy="lfu")
    _parity(w, label=f"c{cid}-lfu-w{ways}")


# ----------------------------------------------------------------------------- random call sequences

@pytest.mark.parametrize("seed,overlap,mode", [(s, True, "zero_copy") for s in range(9)]
                         + [(s, False, "zero_copy") for s in range(6)]
                         + [(s, True, "staged") for s in (0, 1, 2, 4)]
                         + [(s, True, ["zero_copy", "staged", "staged"]) for s in (3, 5)])
def test_random_call_sequences(seed, overlap, mode):
    """Random interleavings of placements and forwards on three streams (two
    placements or two forwards in a row, batches out of order, calls on a
    stream other than the previous call's), checked against the oracle
    replaying the same calls: totals, resident sets and digests at random
    check points, every forward's pooled sums at the end.  The library orders
    calls across streams by events; nothing here synchronises between calls.
    overlap=False: no copy stream, so each fill runs on its placement's stream.
    STAGED and mixed modes: host-gathered rows (prefetch rows gathered while the
    placement ranks) under the same interleavings."""
    import torch as th
    import oracle
    rng = np.random.default_rng(7000 + seed)
    policy = ("lru", "priority", "lfu")[seed % 3]
    w = tg.random_tiny(700 + seed, max_rows=3000, max_cap=300, max_dim=33, batches=10, bags=40,
                       integer_values=False, policy=policy)
    w.ways = (0, 4, 32)[(seed // 3) % 3]
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    o = oracle.for_workload(w, tabs)
    if not isinstance(mode, str):
        mode = (mode * w.num_tables)[:w.num_tables]
    g = GpuRunner(w, tabs, overlap=overlap, miss_mode=mode)
    f64 = [tg.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
    streams = [th.cuda.current_stream(), th.cuda.Stream(), th.cuda.Stream()]
    T = w.num_tables
    tot = [dict() for _ in range(T)]
    outs = []
    last_fwd = None
    from _helpers import FWD_KEYS, PLACE_KEYS

    def add(group, keys):
        for t in range(T):
            st = o.stats(t)
            for k in keys:
                if k != "digest":
                    tot[t][k] = tot[t].get(k, 0) + st[k]

    try:
        for step in range(40):
            op = rng.choice(["plc", "fwd", "plc", "fwd", "check"])
            s = streams[int(rng.integers(3))]
            k = int(rng.integers(w.batches))
            if op == "plc":
                P, poff = w.prefetch_list(k)
                bits = w.cache_bits(last_fwd) if last_fwd is not None else None
                with th.cuda.stream(s):
                    g.cache.placement(g.to_dev(P) if P.size else None, g.to_dev(poff),
                                      None if bits is None else g.to_dev(bits), stream=s)
                assert o.placement(P, poff, bits) == 0
                add("plc", PLACE_KEYS)
            elif op == "fwd":
                idx, off = w.batch(k)
                with th.cuda.stream(s):
                    out = g.cache.forward(g.to_dev(idx), g.to_dev(off), w.bags, stream=s)
                st, _, r64 = o.forward(idx, off, w.bags, want64=True)
                assert st == 0
                add("fwd", FWD_KEYS)
                outs.append((out, r64.copy(), idx, off, step))
                last_fwd = k
            else:
                _, gt, res = g.cache.stats(dump=True)
                for t in range(T):
                    for key, v in tot[t].items():
                        assert gt[t][key] == v, f"step {step} table {t} total {key}"
                    assert np.array_equal(res[t], o.resident(t)), f"step {step} table {t}: resident set"
                    assert gt[t]["digest"] == o.stats(t)["digest"]
        _, gt, res = g.cache.stats(dump=True)
        for t in range(T):
            for key, v in tot[t].items():
                assert gt[t][key] == v, f"end table {t} total {key}"
            assert np.array_equal(res[t], o.resident(t))
        for out, r64, idx, off, step in outs:
            check_pooled(w, f64, idx, off, out.cpu().numpy(), r64, f"forward at step {step}")
    finally:
        g.close()
        o.close()
