#!/usr/bin/env python3
"""Throughput of the tiered pooled-embedding lookup on one MI355X.

One step = one placement (prefetch list + caching bits applied to the HBM
cache) followed by one pooled lookup of a batch, i.e. every row of the hot
path.  Default workload: configuration 5, the one with the most work per batch
-- 64 fp32 tables x 2,000,000 rows with dims 32/64/128/256 (61.4 GB in pinned
host memory), a 200,000-row HBM cache per table, 8,192 bags per table with
geometric(mean 25) pooling (one-hot for the last 16 tables), Zipf exponents
0.8/1.0/1.2, a prefetch list of twice the cache headroom with half of it
precise, PRIORITY ranking (eviction speed 4).  Inputs are synthetic (tracegen)
and resident in HBM before the timed region.

Prints one JSON line: pooled lookups/s (value); the roofline of the kernel
that dominates the step (the fill or the miss fetch, host-link bound) and of
the pooled kernel (HBM bound); host-link traffic; on-demand fetches per batch;
and the CPU oracle timed on the host (cpu_baseline).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PCIE5_X16_GBS = 64.0  # PCIe Gen5 x16, one direction, published
DEFAULT_CONFIG = 5
# HBM bytes per launch of each kernel from rocprofv3 FETCH_SIZE / WRITE_SIZE
# runs of a workload's bench.py command, scaled by a copy-kernel calibration;
# valid only for the kernel source they were measured on (sha256 of the file
# that holds the kernel and of the shared device headers)
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "traffic_config{}.json")
CSRC = os.path.join(ROOT, "paper_2511_08568_amd", "csrc")
KERNEL_FILES = {"pooled": "forward.hip", "k_fetch": "forward.hip", "k_plc_fill": "placement.hip"}
SHARED_HEADERS = ("recmg_device.h", "launch.h")


def kernel_source_sha256(kernel):
    h = hashlib.sha256()
    for f in (KERNEL_FILES[kernel],) + SHARED_HEADERS:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(args, kernel):
    """(bytes per launch, source) of `kernel` when the committed counter record
    matches this workload and the current kernel sources, else (None, reason)."""
    default = (args.row_scale == 1.0 and args.prefetch is None and args.miss_mode == "zero_copy" and args.ways == 0
               and args.bits is None and args.policy is None and args.start_batch == 0 and args.warm_placements == 0)
    if not default:
        return None, "counters recorded for the configurations' own settings only"
    path = TRAFFIC_RECORD.format(args.config)
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None, "no counter record for this configuration"
    k = rec["kernels"].get(kernel)
    if k is None:
        return None, f"{kernel} not in the counter record"
    if k.get("source_sha256") != kernel_source_sha256(kernel):
        return None, "kernel source changed since the counters were taken"
    return (k["read_bytes_per_launch"] + k["write_bytes_per_launch"],
            f"{os.path.relpath(path, ROOT)}: FETCH_SIZE x {rec['fetch_scale']:.2f} + WRITE_SIZE x "
            f"{rec['write_scale']:.2f}, bytes per launch ({k['read_bytes_per_launch'] / 1e6:.1f} MB read, "
            f"{k['write_bytes_per_launch'] / 1e6:.1f} MB written)")


def huge_page_tensor(shape, dtype):
    """Pageable host tensor on transparent 2 MB pages where the kernel offers
    them (madvise mode): the STAGED host gather reads rows at random, and small
    pages would cost a TLB miss per row."""
    import mmap

    import numpy as np
    import torch
    nbytes = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    buf = mmap.mmap(-1, max(nbytes, 1), flags=mmap.MAP_PRIVATE | mmap.MAP_ANONYMOUS)
    if hasattr(mmap, "MADV_HUGEPAGE"):
        try:
            buf.madvise(mmap.MADV_HUGEPAGE)
        except OSError:
            pass
    arr = np.frombuffer(buf, dtype=np.uint8, count=nbytes)
    return torch.from_numpy(arr).view(dtype).view(shape)


_PINNED = []


def pinned_tensor(shape, dtype):
    """Page-locked host tensor of exactly its size, from hipHostMalloc in the
    HIP runtime torch has loaded (torch's pinned allocator rounds a request up
    to a power of two: a 25.6 GB table would pin 32 GiB, and the host caps
    pinned memory).  Freed at exit."""
    import atexit
    import ctypes

    import numpy as np
    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")
    nbytes = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    ptr = ctypes.c_void_p()
    rc = hip.hipHostMalloc(ctypes.byref(ptr), ctypes.c_size_t(max(nbytes, 1)), ctypes.c_uint(0))
    if rc != 0 or not ptr.value:
        raise MemoryError(f"hipHostMalloc of {nbytes} bytes failed with status {rc}")
    if not _PINNED:
        atexit.register(lambda: [hip.hipHostFree(p) for p in _PINNED])
    _PINNED.append(ptr)
    arr = np.ctypeslib.as_array((ctypes.c_uint8 * max(nbytes, 1)).from_address(ptr.value))[:nbytes]
    return torch.from_numpy(arr).view(dtype).view(shape)


def buffer_sweep(args, dev):
    """Hit rate against buffer size on one configuration's trace (Sec. VII-D's
    sweep, on synthetic traces): every point runs the HIP path and the oracle
    on the same batches and checks that their counters agree."""
    import numpy as np
    import torch

    import oracle
    import tracegen as tg
    from paper_2511_08568_amd import TieredEmbeddingCache

    base = tg.make_config(args.config)
    NB = min(args.sweep_batches, base.batches)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.uint16}
    host = [torch.empty((tb.rows, tb.dim), dtype=tdt[tb.dtype], pin_memory=True) for tb in base.tables]
    for t in range(base.num_tables):
        base.table_values(t, out=host[t].numpy())
    tabs_np = [h.numpy() for h in host]
    batches = [base.batch(b) for b in range(NB)]
    seen = [np.unique(np.concatenate([base.uniques(b)[t] for b in range(NB)])).size for t in range(base.num_tables)]
    uniq_total = sum(int(base.uniques(b)[t].size) for b in range(NB) for t in range(base.num_tables))
    recipe = base.prefetch if base.prefetch[0] != "none" else ("exact",)
    # (policy, prefetch recipe, ways): fully associative, and 32-way sets as in
    # the production buffer the paper compares against
    variants = {"lru": ("lru", ("none",), 0), "caching_model": ("priority", ("none",), 0),
                "caching_and_prefetch": ("priority", recipe, 0), "lru_32way": ("lru", ("none",), 32),
                "lfu_32way": ("lfu", ("none",), 32), "caching_and_prefetch_32way": ("priority", recipe, 32)}
    points = []
    for frac in (0.01, 0.02, 0.05, 0.10, 0.15, 0.20, 0.30):
        caps = [max(1, int(round(frac * n))) for n in seen]
        pt = {"buffer_frac_of_touched_rows": frac, "cache_rows": sum(caps)}
        # Belady bound for a demand-filled buffer of Cap rows (no prefetch)
        opt = 0
        for t in range(base.num_tables):
            lab = tg.optgen_labels([base.uniques(b)[t] for b in range(NB)], caps[t])
            opt += sum(int(x.sum()) for x in lab)
        pt["belady_bound"] = opt / uniq_total
        parity = True
        for name, (policy, pf, ways) in variants.items():
            w = tg.make_config(args.config)
            w.policy, w.prefetch, w.ways = policy, pf, ways
            w.bits = ("optgen", 0.8, NB)
            for tb, c in zip(w.tables, caps):
                tb.cap = c
            pre = [w.prefetch_list(b) for b in range(NB)]
            bits = [w.cache_bits(b - 1) if b > 0 else None for b in range(NB)]
            max_idx = max(i.size for i, _ in batches)
            max_pf = max(max(P.size for P, _ in pre), 1)
            cache = TieredEmbeddingCache(host, [tb.dtype for tb in w.tables], caps, policy=policy,
                                         eviction_speed=w.eviction_speed, max_bags_per_table=w.bags,
                                         max_indices=max_idx, max_prefetch=max_pf, ways=ways)
            o = oracle.for_workload(w, tabs_np)
            out = torch.empty(w.bags * sum(tb.dim for tb in w.tables), dtype=torch.float32, device=dev)
            osum = {"hits": 0, "misses": 0, "evicted": 0, "prefetch_fill": 0}
            for b in range(NB):
                P, po = pre[b]
                cache.placement(torch.from_numpy(P).to(dev) if P.size else None, torch.from_numpy(po).to(dev),
                                None if bits[b] is None else torch.from_numpy(bits[b]).to(dev))
                i, off = batches[b]
                cache.forward(torch.from_numpy(i).to(dev), torch.from_numpy(off).to(dev), w.bags, out=out)
                assert o.placement(P, po, bits[b]) == 0
                for t in range(w.num_tables):
                    st = o.stats(t)
                    osum["evicted"] += st["evicted"]
                    osum["prefetch_fill"] += st["prefetch_fill"]
                assert o.forward(i, off, w.bags)[0] == 0
                for t in range(w.num_tables):
                    st = o.stats(t)
                    osum["hits"] += st["hits"]
                    osum["misses"] += st["misses"]
            _, tot = cache.stats()
            cache.close()
            o.close()
            gsum = {k: sum(tot[t][k] for t in range(w.num_tables)) for k in osum}
            parity &= gsum == osum
            pt[name] = gsum["hits"] / uniq_total
            pt[name + "_prefetch_fills"] = gsum["prefetch_fill"]
        pt["counters_equal_oracle"] = parity
        points.append(pt)
        log(f"buffer {frac:.2f}: " + json.dumps({k: round(v, 4) for k, v in pt.items() if isinstance(v, float)}))
    print(json.dumps({"metric": "hit rate (hits / distinct rows per batch, summed) vs buffer size",
                      "workload": describe_workload(args.config, base), "batches": NB,
                      "caching_bits": "OPTgen labels for a buffer of 0.8 x Cap over the same batches",
                      "prefetch_recipe": list(recipe), "points": points}), flush=True)


def describe_workload(cid, w):
    """One line naming the configuration by its shapes."""
    tabs = w.tables

    def span(vals, fmt="{:,}"):
        lo, hi = min(vals), max(vals)
        return fmt.format(lo) if lo == hi else f"{fmt.format(lo)}..{fmt.format(hi)}"

    dims = sorted({tb.dim for tb in tabs})
    pools = sorted({tb.pooling[0] for tb in tabs})
    return (f"configuration {cid}: {len(tabs)} {'/'.join(sorted({tb.dtype for tb in tabs}))} tables, "
            f"{span([tb.rows for tb in tabs])} rows x dim {'/'.join(map(str, dims))}, "
            f"HBM cache {sum(tb.cap for tb in tabs):,} rows in all, {w.bags:,} bags/table, "
            f"pooling {'/'.join(pools)} (table 0: {tabs[0].pooling}), "
            f"Zipf {span([tb.alpha for tb in tabs], '{:.2f}')}, prefetch {w.prefetch}, policy {w.policy}"
            + (f", {w.ways}-way sets" if w.ways else ""))


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=DEFAULT_CONFIG, help="configuration id (1..5)")
    ap.add_argument("--row-scale", type=float, default=1.0, help="<1 shrinks rows and caches (debug only)")
    ap.add_argument("--miss-mode", default="zero_copy", choices=["zero_copy", "staged"])
    ap.add_argument("--zero-copy-tables", type=int, default=0, metavar="N",
                    help="with --miss-mode staged: the first N tables pinned and read zero-copy, the rest "
                         "gathered on the host (for tables that do not all fit the host's pinned-memory limit)")
    ap.add_argument("--prefetch", default=None, choices=["none", "exact"],
                    help="override the configuration's prefetch recipe (configuration 4 is run both ways)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="time budget of the CPU oracle sample")
    ap.add_argument("--breakdown-steps", type=int, default=10,
                    help="steps after the timed ones with every stage timed (stage split, host-link rate)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-link-peak", action="store_true")
    ap.add_argument("--bits", default=None, choices=["lookahead", "optgen"],
                    help="caching-bit source of PRIORITY configurations (optgen: Belady-optimal labels for a "
                         "buffer of 0.8 x Cap over the run's batches)")
    ap.add_argument("--buffer-sweep", action="store_true",
                    help="instead of the benchmark: hit rate against buffer size (1-30%% of the rows the trace "
                         "touches) for LRU, the caching policy with OPTgen bits, that policy with the "
                         "configuration's prefetch list, and the Belady bound; one JSON line")
    ap.add_argument("--sweep-batches", type=int, default=60)
    ap.add_argument("--no-pipeline", dest="pipeline", action="store_false",
                    help="run placements on the forward's stream (no overlap of placement b+1 with forward b)")
    ap.add_argument("--no-copy-stream", dest="copy_stream", action="store_false",
                    help="ZERO_COPY: run the prefetch fill on the placement's stream, not a copy stream of its "
                         "own (with --no-pipeline every kernel of a step is on one stream: no cross-stream waits, "
                         "which a launch-bound small batch feels)")
    ap.add_argument("--policy", default=None, choices=["lru", "priority", "lfu"],
                    help="override the configuration's placement policy")
    ap.add_argument("--ways", type=int, default=0,
                    help="W > 0: W-way set-associative caches (Alg. 2 inside each set) instead of fully "
                         "associative ones")
    ap.add_argument("--start-batch", type=int, default=0,
                    help="play the trace from this batch on (with --warm-placements: a cache in steady state)")
    ap.add_argument("--warm-placements", type=int, default=0, metavar="N",
                    help="before the warmup steps, N placements with no forward between them whose prefetch lists "
                         "name each table's Cap most popular rows, so the caches start full")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 3 device-to-device copies of MIB MiB (scale for HBM byte counters) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU: each configuration's tables are one GPU's "
                                   "share (sharding by table is described, not built); --gpus must be 1"}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import tracegen as tg
    from paper_2511_08568_amd import TieredEmbeddingCache

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        a = torch.ones(n, dtype=torch.uint8, device=dev)
        z = torch.empty_like(a)
        for _ in range(3):
            z.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 3}), flush=True)
        return
    if args.buffer_sweep:
        buffer_sweep(args, dev)
        return
    if args.row_scale < 1.0:
        w = tg.scaled_config(args.config, row_scale=args.row_scale)
    else:
        w = tg.make_config(args.config)
    if args.prefetch is not None:
        w.prefetch = (args.prefetch,)
    w.ways = args.ways
    if args.policy is not None:
        w.policy = args.policy
    W, K, S0, NW = args.warmup, args.steps, args.start_batch, args.warm_placements
    if S0 < 0 or NW < 0 or S0 + W + K > w.batches:
        raise SystemExit(f"start + warmup + steps must be at most the workload's {w.batches} batches")
    # after the timed steps, a few more with every stage timed (the breakdown)
    KB = min(args.breakdown_steps, w.batches - S0 - W - K)
    nb = W + K + KB
    if args.bits == "optgen":
        w.bits = ("optgen", 0.8, nb + 1)  # labels over the batches this run plays
    T = w.num_tables

    # -- tables in pinned host memory -------------------------------------------------------------
    t0 = time.time()
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.uint16}
    # zero-copy tables are pinned (the GPU reads them); STAGED tables are read
    # on the host only and stay pageable
    modes = ["zero_copy" if args.miss_mode == "zero_copy" or t < args.zero_copy_tables else "staged"
             for t in range(T)]
    host = [pinned_tensor((tb.rows, tb.dim), tdt[tb.dtype]) if m == "zero_copy"
            else huge_page_tensor((tb.rows, tb.dim), tdt[tb.dtype]) for tb, m in zip(w.tables, modes)]
    for t in range(T):  # each table's rows are drawn in parallel chunks
        w.table_values(t, out=host[t].numpy())
    log(f"tables ready ({sum(h.numel() * h.element_size() for h in host) / 1e9:.2f} GB, "
        f"{modes.count('zero_copy')} of {T} pinned) in {time.time() - t0:.1f}s")

    # -- traces, staged into HBM before timing ----------------------------------------------------
    t0 = time.time()
    # step b plays batch S0 + b; the caching bits of its placement come from
    # the batch before it, if this run played that batch
    batches, prefetch, bits = [], [], []
    for b in range(nb):
        idx, off = w.batch(S0 + b)
        P, poff = w.prefetch_list(S0 + b)
        cb = w.cache_bits(S0 + b - 1) if b > 0 else None
        batches.append((idx, off))
        prefetch.append((P, poff))
        bits.append(cb)
    warm_lists = [w.warm_list(k, NW) for k in range(NW)]
    d_warm = [(torch.from_numpy(P).to(dev), torch.from_numpy(po).to(dev)) for P, po in warm_lists]
    d_batches = [(torch.from_numpy(i).to(dev), torch.from_numpy(o).to(dev)) for i, o in batches]
    d_prefetch = [(torch.from_numpy(P).to(dev) if P.size else None, torch.from_numpy(po).to(dev))
                  for P, po in prefetch]
    d_bits = [None if cb is None else torch.from_numpy(cb).to(dev) for cb in bits]
    max_idx = max(i.size for i, _ in batches)
    max_pf = max(max(P.size for P, _ in prefetch + warm_lists), 1)
    # one output buffer per batch, so that every batch can be checked against the oracle afterwards
    outs = [torch.empty(w.bags * sum(tb.dim for tb in w.tables), dtype=torch.float32, device=dev) for _ in range(nb)]
    torch.cuda.synchronize()
    log(f"{nb} batches staged in {time.time() - t0:.1f}s (max {max_idx} indices)")

    cache = TieredEmbeddingCache(host, [tb.dtype for tb in w.tables], [tb.cap for tb in w.tables], policy=w.policy,
                                 eviction_speed=w.eviction_speed, miss_mode=modes,
                                 max_bags_per_table=w.bags, max_indices=max_idx, max_prefetch=max_pf, timing=1,
                                 ways=w.ways, stats_log_calls=2 * nb + NW, overlap=args.copy_stream)
    log(f"cache ready: workspace {cache.workspace_bytes / 1e9:.2f} GB")

    # Pipelined placement: placements run on a stream of their own, so that
    # placement b+1 (which needs forward b's distinct rows and misses) overlaps
    # forward b's fill wait and pooled kernel; the library orders the two
    # streams with events.  Inputs are already on the device.
    pstream = torch.cuda.Stream(device=dev) if args.pipeline else None

    def step(b, marks=None):
        P, po = d_prefetch[b]
        cache.placement(P, po, d_bits[b], stream=pstream)
        if marks is not None:
            marks[b].record(pstream if pstream is not None else torch.cuda.current_stream())
        i, o = d_batches[b]
        cache.forward(i, o, w.bags, out=outs[b])

    if NW:
        t0 = time.time()
        for P, po in d_warm:
            cache.placement(P, po, None, stream=pstream)
        torch.cuda.synchronize()
        log(f"{NW} warm-up placements in {time.time() - t0:.1f}s: "
            f"{sum(r['resident'] for r in cache.stats()[0]):,} rows resident")
    for b in range(W):
        step(b)
    torch.cuda.synchronize()
    _, tot0 = cache.stats()
    cache.stage_times(reset=True)

    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    if pstream is not None:
        pstream.wait_event(ev0)
    for b in range(W, W + K):
        step(b)
    ev1.record(stream)  # after the last forward, which waited for every placement and fill
    torch.cuda.synchronize()
    elapsed_ms = ev0.elapsed_time(ev1)
    timed_stages = cache.stage_times(reset=True)  # the pooled kernel only (timing level 1)
    _, tot1 = cache.stats()
    log(f"timed {K} steps: {elapsed_ms:.3f} ms; kernels (ms): pooled {timed_stages['fwd_pool'][0]:.3f}, "
        f"fill {timed_stages['plc_fill'][0]:.3f}, fetch {timed_stages['fwd_fetch'][0]:.3f}, "
        f"host-link union {timed_stages['host_link'][0]:.3f}")
    # breakdown: every stage timed (each stage adds two stream commands, so
    # these steps are slower and stay out of the headline figure)
    # Events before each placement and between it and its forward also split
    # the step into placement and forward time (the forward's share includes
    # waiting for the placement's prefetch fill on the side stream).
    stages, tot2, plc_ms, fwd_ms = timed_stages, tot1, 0.0, 0.0
    if KB > 0:
        cache.set_timing(2)
        marks = {b: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for b in range(W + K, nb)}
        end = torch.cuda.Event(enable_timing=True)
        for b in range(W + K, nb):
            marks[b][0].record(stream)
            if pstream is not None:
                pstream.wait_event(marks[b][0])  # the split needs the placement between the two marks
            step(b, {b: marks[b][1]})
        end.record(stream)
        torch.cuda.synchronize()
        plc_ms = sum(marks[b][0].elapsed_time(marks[b][1]) for b in range(W + K, nb))
        fwd_ms = sum(marks[b][1].elapsed_time(marks[b + 1][0] if b + 1 < nb else end) for b in range(W + K, nb))
        stages = cache.stage_times(reset=True)
        _, tot2 = cache.stats()
        log(f"breakdown over {KB} steps: {json.dumps({k: round(v[0], 3) for k, v in stages.items()})}")

    # -- metrics ---------------------------------------------------------------------------------
    lookups = sum(int(batches[b][0].size) for b in range(W, W + K))
    delta = {k: sum(tot1[t][k] - tot0[t][k] for t in range(T)) for k in tot1[0] if k != "digest"}
    pool_ms, pool_calls = timed_stages["fwd_pool"]
    # Bytes of one pooled launch.  Algorithmic minimum: every distinct row of the
    # batch read once (repeats need not come from HBM again), a 4-byte location
    # per index, an 8-byte offset and the fp32 output per bag.  Logical: a full
    # row per index.
    alg_bytes, logical_bytes = 0, 0
    for t, tb in enumerate(w.tables):
        alg_bytes += (tot1[t]["unique"] - tot0[t]["unique"]) * tb.row_bytes
    for b in range(W, W + K):
        idx, off = batches[b]
        for t, tb in enumerate(w.tables):
            s, e = w.table_segment(off, t)
            per_bag = w.bags * (8 + 4 * tb.dim)
            alg_bytes += (e - s) * 4 + per_bag
            logical_bytes += (e - s) * (tb.row_bytes + 4) + per_bag
    bytes_per_launch = alg_bytes / K
    pool_s = pool_ms / max(pool_calls, 1) / 1e3
    achieved = bytes_per_launch / pool_s / 1e9 if pool_s > 0 else 0.0
    # The host-link kernels over the timed steps, by the events their own
    # dispatches record (timing level 1): the placement's fill (prefetch rows
    # read from pinned host memory; admitted misses come from HBM staging) and
    # the forward's zero-copy miss fetch.  They run at the same time on two
    # streams, so each kernel's own rate is its share of the link; the union
    # of their intervals gives the link's rate.
    fill_ms, fill_calls = timed_stages["plc_fill"]
    fetch_ms, fetch_calls = timed_stages["fwd_fetch"]
    union_ms = timed_stages["host_link"][0]
    host_bytes = {"k_plc_fill": delta["prefetch_bytes"], "k_fetch": delta["ondemand_bytes"]}
    link_times = {"k_plc_fill": (fill_ms, fill_calls), "k_fetch": (fetch_ms, fetch_calls)}
    zero_copy = all(m == "zero_copy" for m in modes)
    # host link over the breakdown steps: bytes moved there / the union of the
    # miss-fetch and fill intervals (they overlap on two streams)
    bdelta = {k: sum(tot2[t][k] - tot1[t][k] for t in range(T)) for k in tot2[0] if k != "digest"}
    link_bytes = bdelta["ondemand_bytes"] + bdelta["prefetch_bytes"]
    link_ms = stages["host_link"][0]
    link_gbs = link_bytes / (link_ms / 1e3) / 1e9 if link_ms > 0 else 0.0

    pool_traffic, pool_tsrc = measured_traffic(args, "pooled")

    link_peak = None
    if not args.no_link_peak:
        buf = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
        dbuf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        best = 0.0
        for _ in range(10):
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dbuf.copy_(buf, non_blocking=True)
            z.record()
            torch.cuda.synchronize()
            best = max(best, (1 << 30) / (a.elapsed_time(z) / 1e3) / 1e9)
        link_peak = best
        del buf, dbuf

    result = {
        "metric": "pooled lookups/s",
        "value": lookups / (elapsed_ms / 1e3),
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": elapsed_ms / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",  # sums accumulate in fp32 whatever the storage type
        "storage_dtype": sorted({tb.dtype for tb in w.tables}),
        "data": "synthetic (seeded Zipf traces standing in for the paper's Meta embedding-lookup traces)",
        "config": {
            "workload": describe_workload(args.config, w),
            "batches": (f"{NW} warm-up placements filling the caches, then " if NW else "")
                       + f"batches {S0}.. : {W} warmup + {K} timed, each placement + forward",
            "miss_mode": args.miss_mode if len(set(modes)) == 1 else
                         f"mixed: tables 0..{args.zero_copy_tables - 1} zero_copy, the rest staged",
            "pipelined_placement": bool(args.pipeline),
            "copy_stream": bool(args.copy_stream or args.miss_mode == "staged"),
            "row_scale": args.row_scale,
        },
        "hit_path_roofline": {
            "kernel": "k_pool_w (pooled gather + sum; one launch per row-size kind, timed together per forward)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": pool_traffic,
            "traffic_source": pool_tsrc,
            "alg_bytes_per_launch": bytes_per_launch,
            "avg_launch_us": pool_s * 1e6,
            "logical_bytes_per_launch": logical_bytes / K,
            "logical_GBs": logical_bytes / K / pool_s / 1e9 if pool_s > 0 else 0.0,
        },
        "split": {"placement_ms_per_step": plc_ms / max(KB, 1), "forward_ms_per_step": fwd_ms / max(KB, 1),
                  "forward_only_lookups_per_s": (sum(int(batches[b][0].size) for b in range(W + K, nb)) / (fwd_ms / 1e3)
                                                 if fwd_ms > 0 else None),
                  "measured_over": f"{KB} breakdown steps (every stage timed; with pipelined placement "
                                   "each breakdown placement starts after the previous forward, so the two "
                                   "do not overlap there)"},
        "ondemand_fetches_per_batch": delta["misses"] / K,
        # Sec. IV Eq. coverage (unique vectors of the batch the list names) and
        # prefetch accuracy (of the distinct rows prefetched, those the batch
        # uses), over the timed steps
        "prefetch_quality": {"coverage": delta["prefetch_covered"] / max(delta["unique"], 1),
                             "accuracy": (delta["prefetch_covered"] / delta["prefetch_distinct"]
                                          if delta["prefetch_distinct"] else None),
                             "prefetch_distinct_per_batch": delta["prefetch_distinct"] / K},
        "prefetch_fills_per_batch": delta["prefetch_fill"] / K,
        "host_link": {"bytes_per_batch": link_bytes / max(KB, 1), "achieved_GBs": link_gbs,
                      "measured_over": f"{KB} breakdown steps after the timed ones",
                      "measured_h2d_peak_GBs": link_peak, "pcie5_x16_GBs": PCIE5_X16_GBS,
                      "frac_of_measured_peak": (link_gbs / link_peak) if link_peak else None},
        "hit_rate": delta["hits"] / max(delta["unique"], 1),
        "stage_ms_per_step": {k: v[0] / max(KB, 1) for k, v in stages.items()},
        "stage_split_over": f"{KB} breakdown steps (every stage timed) after the timed ones",
    }

    # The roofline object describes the kernel that takes most of the timed
    # steps' kernel time.  With zero-copy misses that is the fill or the miss
    # fetch whenever either moves more than a few MB per batch: they are bound
    # by the host link (PCIe Gen5 x16), not by HBM, and are priced against it.
    link_kernel = max(link_times, key=lambda k: link_times[k][0])
    if zero_copy and link_times[link_kernel][0] > pool_ms:
        ms, calls = link_times[link_kernel]
        avg_s = ms / max(calls, 1) / 1e3
        per_launch = host_bytes[link_kernel] / max(calls, 1)
        ach = per_launch / avg_s / 1e9 if avg_s > 0 else 0.0
        traffic, tsrc = measured_traffic(args, link_kernel)
        union_gbs = sum(host_bytes.values()) / (union_ms / 1e3) / 1e9 if union_ms > 0 else 0.0
        result["roofline"] = {
            "kernel": link_kernel + (" (prefetch fill: host rows into HBM slots)" if link_kernel == "k_plc_fill"
                                     else " (zero-copy on-demand miss fetch)"),
            "bound": "host_link",
            "achieved": ach,
            "peak": PCIE5_X16_GBS,
            "unit": "GB/s",
            "frac": ach / PCIE5_X16_GBS,
            "traffic": traffic,
            "traffic_source": tsrc,
            "alg_bytes_per_launch": per_launch,
            "avg_launch_us": avg_s * 1e6,
            "frac_of_measured_peak": ach / link_peak if link_peak else None,
            "measured_h2d_peak_GBs": link_peak,
            "link_shared_with": ("k_fetch" if link_kernel == "k_plc_fill" else "k_plc_fill") + " on the other stream",
            "link_union": {"bytes_per_step": sum(host_bytes.values()) / K,
                           "ms_per_step": union_ms / K,
                           "achieved_GBs": union_gbs,
                           "frac": union_gbs / PCIE5_X16_GBS,
                           "frac_of_measured_peak": union_gbs / link_peak if link_peak else None},
        }
    else:
        result["roofline"] = dict(result["hit_path_roofline"])

    # what the oracle replay checks: every call's counters (the device log),
    # the final resident sets, and the pooled sums of every batch, or of a
    # fixed subset (every 5th, the first and the last) where checking all would
    # take the host too long
    call_log = cache.stats_log()
    _, _, final_res = cache.stats(dump=True)
    work = sum(int(batches[b][0].size) for b in range(nb)) * (sum(tb.dim for tb in w.tables) / T)
    check = list(range(nb)) if work <= 1e10 else sorted({0, nb - 1, *range(0, nb, 5)})
    gpu_out = {b: outs[b].cpu().numpy() for b in check}
    del outs
    cache.close()

    if not args.no_cpu_baseline:
        # The oracle replays the same batches on the host: timed as the CPU
        # baseline, and compared with the GPU run (every call's counters and
        # digest, the totals, the final resident sets, the checked batches'
        # pooled sums against rtol x L1 mass).
        import oracle
        cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
        nth = max(1, min(cores, T))
        tabs_np = [h.numpy() for h in host]
        o = oracle.for_workload(w, tabs_np, nthreads=nth)
        sums = [dict.fromkeys(tot1[0], 0) for _ in range(T)]
        # The timed sample is the replay of the GPU's batches (always whole, for
        # the parity check), continued with the workload's next batches
        # (generated outside the timed intervals) until about --cpu-seconds of
        # oracle time.
        done, n_lookups, secs = 0, 0, 0.0
        calls_equal, digests_equal, res_equal, pooled_ok, worst = True, True, None, True, 0.0
        # output buffers allocated once, outside the timed intervals
        n_out = w.bags * sum(tb.dim for tb in w.tables)
        o32, o64 = np.zeros(max(n_out, 1), np.float32), np.zeros(max(n_out, 1), np.float64)
        rtol = {"f32": 1e-5, "f16": 2e-2, "bf16": 2e-2}
        # the warm-up placements (untimed): calls 0 .. NW - 1 of the device log
        for k, (P, poff) in enumerate(warm_lists):
            assert o.placement(P, poff, None) == 0
            for t in range(T):
                st = o.stats(t)
                for key in oracle.PLC_FIELDS:
                    calls_equal &= call_log[k][t][key] == st[key]
                    sums[t][key] += st[key]
                digests_equal &= call_log[k][t]["digest"] == st["digest"]
        last_log = time.time()
        for b in range(w.batches - S0):
            if time.time() - last_log > 15:
                log(f"oracle: batch {b}, {secs:.1f}s of oracle time")
                last_log = time.time()
            if b < nb:
                (P, poff), cb, (idx, off) = prefetch[b], bits[b], batches[b]
            elif secs > args.cpu_seconds:
                break
            else:
                P, poff = w.prefetch_list(S0 + b)
                cb = w.cache_bits(S0 + b - 1)
                idx, off = w.batch(S0 + b)
            t_start = time.time()
            assert o.placement(P, poff, cb) == 0
            secs += time.time() - t_start
            plc = [o.stats(t) for t in range(T)] if b < nb else None
            t_start = time.time()
            st, _, r64 = o.forward(idx, off, w.bags, out32=o32, out64=o64 if b in gpu_out else None)
            secs += time.time() - t_start
            assert st == 0
            if b < nb:
                # this batch's two calls against the device log: placement NW + 2b, forward NW + 2b + 1
                for t in range(T):
                    fw = o.stats(t)
                    for k in oracle.PLC_FIELDS:
                        calls_equal &= call_log[NW + 2 * b][t][k] == plc[t][k]
                    for k in oracle.FWD_FIELDS:
                        calls_equal &= call_log[NW + 2 * b + 1][t][k] == fw[k]
                    digests_equal &= call_log[NW + 2 * b][t]["digest"] == plc[t]["digest"]
                if b in gpu_out:
                    mass = o.pooled_abs(idx, off, w.bags)  # the tolerance scale, outside the timed intervals
                    err = np.abs(gpu_out[b].astype(np.float64) - r64)
                    at = 0
                    for t, tb in enumerate(w.tables):
                        n = w.bags * tb.dim
                        pooled_ok &= bool(np.all(err[at:at + n] <= rtol[tb.dtype] * mass[at:at + n]))
                        at += n
                    worst = max(worst, float((err / np.maximum(mass, 1e-300)).max()) if err.size else 0.0)
                if b == nb - 1:
                    res_equal = all(np.array_equal(final_res[t], o.resident(t)) for t in range(T))
            if b < nb:
                for t in range(T):
                    fw = o.stats(t)
                    for k in sums[t]:
                        if k == "digest":
                            sums[t][k] = plc[t][k]
                        elif k in oracle.FWD_FIELDS:
                            sums[t][k] += fw[k]
                        else:
                            sums[t][k] += plc[t][k]
            n_lookups += idx.size
            done += 1
        o.close()
        cpu_model = ""
        try:
            with open("/proc/cpuinfo") as fh:
                cpu_model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
        except OSError:
            pass
        result["cpu_baseline"] = {
            "value": n_lookups / secs,
            "unit": "lookups/s",
            "cores": nth,
            "kind": "oracle",
            "sample": f"batches {S0}..{S0 + done - 1} of the same workload (placement + forward each; the first {min(done, nb)} "
                      f"are the GPU run's), {secs:.1f}s of oracle time, {nth} threads (one per table, at most one per "
                      f"usable core)",
            "cpu_model": cpu_model,
        }
        if done >= nb:
            totals_equal = all(sums[t][k] == tot2[t][k] for t in range(T) for k in sums[t] if k != "digest")
            result["parity"] = {
                "batches": nb,
                "counters_equal_every_call": bool(calls_equal and totals_equal),
                "digest_equal_every_placement": bool(digests_equal),
                "final_resident_sets_equal": bool(res_equal),
                "pooled_batches_checked": len(check) if len(check) < nb else "all",
                "pooled_within_tol": bool(pooled_ok),
                "pooled_max_err_over_l1": worst,
            }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
