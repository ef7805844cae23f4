"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each ``pin_*`` function takes the oracle variant to check (``mutant`` 0 is the
real oracle; k > 0 builds it with a planted mistake) and raises AssertionError
on a mismatch.  ``test_oracle_pins.py`` runs them on the real oracle and
``test_oracle_mutants.py`` shows that every planted mistake trips at least one.

Sources of truth used here:
  * hand-worked traces of Sec. VI-B (Alg. 1 / Alg. 2) under the stated readings
    (``tests/golden/hand_*.json``);
  * ``torch.nn.functional.embedding_bag(mode="sum")`` in float64 on the CPU
    (the textbook pooled lookup, Sec. II);
  * the published first outputs of SplitMix64 seeded with 0;
  * closed forms that hold for special cases: an LRU cache keeps the Cap rows
    with the most recent events (global history), an LFU cache the Cap rows
    with the most batches accessed (among rows ever offered), an unbounded cache keeps
    everything it was offered, a zero-capacity cache never hits, and with
    eviction_speed 0 the priority policy reduces to ranking by row id;
  * invariants: hits + misses = distinct rows, |R| <= Cap, resident-count
    conservation, digest = sum of SplitMix64 mixes over the resident dump.
Set-associative caches (ways W > 0) are pinned by three hand-worked traces and:
  * a direct-mapped cache (W = 1) holds, per set, the largest prefetched row of
    the set if any, else the largest missed row, else what it held;
  * LRU_BATCH with one event per set per batch keeps, per set, the W rows with
    the latest events (no ties, so the closed form is exact);
  * when every set can hold all of its rows, nothing is evicted;
  * invariants: at most W residents per set, digest over the dump.
"""
import numpy as np
import torch

import oracle
import tracegen as tg
from _helpers import golden_table, load_golden, splitmix64_mix_py

GOLDEN_FILES = ("hand_lru.json", "hand_priority_es4.json", "hand_priority_es1.json", "hand_priority_es0.json",
                "hand_sa_lru_w2.json", "hand_sa_priority_w2.json", "hand_sa_priority_es1.json",
                "hand_sa_lfu_w2.json")


# ----------------------------------------------------------------------------- drivers

def run_oracle(w, mutant=0, nbatches=None, want64=True):
    """Drive the oracle through ``w``: placement(P_b, bits_{b-1}) then forward(I_b)."""
    T = w.num_tables
    tabs = [w.table_values(t) for t in range(T)]
    o = oracle.for_workload(w, tabs, mutant=mutant)
    recs = []
    for b in range(nbatches or w.batches):
        P, poff = w.prefetch_list(b)
        bits = w.cache_bits(b - 1) if b > 0 else None
        assert o.placement(P, poff, bits) == 0
        place = [o.stats(t) for t in range(T)]
        res = [o.resident(t) for t in range(T)]
        idx, off = w.batch(b)
        st, out32, out64 = o.forward(idx, off, w.bags, want64=want64)
        assert st == 0
        fwd = [o.stats(t) for t in range(T)]
        recs.append(dict(place=place, resident=res, fwd=fwd, out32=out32, out64=out64, P=P, poff=poff,
                         idx=idx, off=off))
    o.close()
    return tabs, recs


def segments(w, off):
    return [w.table_segment(off, t) for t in range(w.num_tables)]


# ----------------------------------------------------------------------------- pins

def pin_hand_examples(mutant=0):
    for name in GOLDEN_FILES:
        g = load_golden(name)
        tab = golden_table(g)
        o = oracle.Oracle([tab], ["f32"], [g["cap"]], policy=g["policy"], eviction_speed=g["eviction_speed"],
                          mutant=mutant, ways=g.get("ways", 0))
        for b, step in enumerate(g["steps"]):
            P = np.array(step["prefetch"], np.int32)
            bits = None if step["bits"] is None else np.array(step["bits"], np.uint8)
            assert o.placement(P, np.array([0, P.size], np.int64), bits) == 0
            s = o.stats(0)
            for k, v in step["expect_placement"].items():
                assert s[k] == v, f"{name} placement {b}: {k} = {s[k]}, hand-worked {v}"
            assert list(o.resident(0)) == step["resident"], f"{name} placement {b}: resident {list(o.resident(0))}"
            idx = np.array(step["indices"], np.int32)
            off = np.array(step["offsets"], np.int64)
            st, out32, _ = o.forward(idx, off, off.size - 1)
            assert st == 0
            s = o.stats(0)
            for k, v in step["expect_forward"].items():
                assert s[k] == v, f"{name} forward {b}: {k} = {s[k]}, hand-worked {v}"
            want = np.array(step["out"], np.float32).reshape(-1)
            assert np.array_equal(out32, want), f"{name} forward {b}: out {out32} != {want}"
        o.close()


def pin_embedding_bag(mutant=0):
    """Pooled sums against torch's embedding_bag(mode='sum') in float64."""
    cases = [tg.random_tiny(s, max_rows=40, max_dim=9, batches=3, bags=5, integer_values=(s % 2 == 0))
             for s in range(12)]
    cases.append(tg.scaled_config(1, row_scale=0.01, batches=2, bags=64))
    for w in cases:
        tabs, recs = run_oracle(w, mutant=mutant)
        f64 = [tg.storage_to_f64(a, tb.dtype) for a, tb in zip(tabs, w.tables)]
        for r in recs:
            ref = []
            for t in range(w.num_tables):
                s, e = w.table_segment(r["off"], t)
                o_t = torch.from_numpy(r["off"][t * w.bags:(t + 1) * w.bags + 1] - s)
                ref.append(torch.nn.functional.embedding_bag(
                    torch.from_numpy(r["idx"][s:e].astype(np.int64)), torch.from_numpy(f64[t]), o_t,
                    mode="sum", include_last_offset=True).numpy().reshape(-1))
            ref = np.concatenate(ref) if ref else np.zeros(0)
            # the L1 mass (tolerance scale) is the pooled sum of |table|
            o2 = oracle.for_workload(w, tabs, mutant=mutant)
            absref = []
            for t in range(w.num_tables):
                s, e = w.table_segment(r["off"], t)
                o_t = torch.from_numpy(r["off"][t * w.bags:(t + 1) * w.bags + 1] - s)
                absref.append(torch.nn.functional.embedding_bag(
                    torch.from_numpy(r["idx"][s:e].astype(np.int64)), torch.from_numpy(np.abs(f64[t])), o_t,
                    mode="sum", include_last_offset=True).numpy().reshape(-1))
            absref = np.concatenate(absref) if absref else np.zeros(0)
            assert np.allclose(o2.pooled_abs(r["idx"], r["off"], w.bags), absref, rtol=1e-12, atol=1e-12)
            o2.close()
            if w.integer_values:
                assert np.array_equal(r["out64"], ref), "integer-valued pooled sums must be exact"
                assert np.array_equal(r["out32"], ref.astype(np.float32))
            else:
                assert np.allclose(r["out64"], ref, rtol=1e-12, atol=1e-12)
                assert np.array_equal(r["out32"], r["out64"].astype(np.float32)), "one rounding of the fp64 sum"


def pin_splitmix(mutant=0):
    """Published first outputs of SplitMix64 seeded with 0: mix(k * golden gamma)."""
    gamma = 0x9E3779B97F4A7C15
    published = (0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC)
    for k, want in enumerate(published, start=1):
        z = (k * gamma) & ((1 << 64) - 1)
        assert oracle.splitmix64_mix(z, mutant) == want
        assert splitmix64_mix_py(z) == want


def pin_lru_history(mutant=0, seeds=range(40)):
    """LRU_BATCH keeps the Cap rows whose most recent event (access in forward f
    -> f, prefetch before forward p -> p) is latest, ties to the higher id.  A
    row admitted while P names it (a miss of the last batch included) is
    flagged until it is accessed (R16)."""
    for s in seeds:
        w = tg.random_tiny(s, policy="lru", batches=6)
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        T = w.num_tables
        last = [dict() for _ in range(T)]
        R = [set() for _ in range(T)]
        pf_live = [dict() for _ in range(T)]
        for b, r in enumerate(recs):
            dig_t = []
            for t in range(T):
                P = set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                for p in P:
                    last[t][p] = max(last[t].get(p, -1), b)
                ranked = sorted(last[t], key=lambda x: (last[t][x], x), reverse=True)
                newR = set(ranked[: w.tables[t].cap])
                for x in newR - R[t]:
                    pf_live[t][x] = x in P
                for x in R[t] - newR:
                    pf_live[t].pop(x, None)
                R[t] = newR
                assert sorted(newR) == r["resident"][t].tolist(), f"seed {s} batch {b} table {t}"
                assert r["place"][t]["resident"] == len(newR)
                dig_t.append(sum(splitmix64_mix_py((t << 40) | x) for x in newR) & ((1 << 64) - 1))
                assert r["place"][t]["digest"] == dig_t[-1], f"seed {s} batch {b} table {t}: digest"
            for t, (a, e) in enumerate(segments(w, r["off"])):
                U = set(r["idx"][a:e].tolist())
                assert r["fwd"][t]["misses"] == len(U - R[t])
                assert r["fwd"][t]["hits"] == len(U & R[t])
                assert r["fwd"][t]["hits_prefetch"] == sum(1 for x in U & R[t] if pf_live[t].get(x))
                for x in U:
                    last[t][x] = b
                    if x in R[t]:
                        pf_live[t][x] = False


def pin_lfu_history(mutant=0, seeds=range(40)):
    """LFU_BATCH keeps the Cap rows with the largest (f, row), f = number of
    batches that accessed the row before this placement, over every row ever
    accessed or prefetched: a row leaves only for Cap rows of larger key, and
    keys never decrease, so it can come back only through a new event."""
    for s in seeds:
        w = tg.random_tiny(s, policy="lfu", batches=6)
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        T = w.num_tables
        f = [dict() for _ in range(T)]
        offered = [set() for _ in range(T)]
        for b, r in enumerate(recs):
            for t in range(T):
                offered[t] |= set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                ranked = sorted(offered[t], key=lambda x: (f[t].get(x, 0), x), reverse=True)
                R = set(ranked[: w.tables[t].cap])
                assert sorted(R) == r["resident"][t].tolist(), f"seed {s} batch {b} table {t}"
            for t, (a, e) in enumerate(segments(w, r["off"])):
                U = set(r["idx"][a:e].tolist())
                assert r["fwd"][t]["misses"] == len(U - set(r["resident"][t].tolist()))
                for x in U:
                    f[t][x] = f[t].get(x, 0) + 1
                offered[t] |= U


def pin_unbounded_cache(mutant=0, seeds=range(20)):
    """Cap >= N: nothing is ever evicted; the cache holds every row accessed or
    prefetched so far, and the misses of a batch are its never-seen rows."""
    for s in seeds:
        w = tg.random_tiny(s, batches=5)
        for tb in w.tables:
            tb.cap = tb.rows
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        seen = [set() for _ in w.tables]
        for b, r in enumerate(recs):
            for t in range(w.num_tables):
                seen[t] |= set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                assert r["resident"][t].tolist() == sorted(seen[t])
                assert r["place"][t]["evicted"] == 0
            for t, (a, e) in enumerate(segments(w, r["off"])):
                U = set(r["idx"][a:e].tolist())
                assert r["fwd"][t]["misses"] == len(U - seen[t])
                seen[t] |= U


def pin_zero_capacity(mutant=0, seeds=range(10)):
    for s in seeds:
        w = tg.random_tiny(s, batches=4)
        for tb in w.tables:
            tb.cap = 0
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        for r in recs:
            for t, (a, e) in enumerate(segments(w, r["off"])):
                U = np.unique(r["idx"][a:e])
                assert r["fwd"][t]["hits"] == 0 and r["fwd"][t]["misses"] == U.size
                assert r["place"][t]["resident"] == 0
                assert r["place"][t]["prefetch_dropped"] == np.unique(r["P"][r["poff"][t]:r["poff"][t + 1]]).size


def pin_priority_es0(mutant=0, seeds=range(30)):
    """eviction_speed 0.  Bits all 0: every score stays 0, so the cache keeps
    the Cap highest ids of R ∪ U_{b-1} ∪ P_b.  Bits all 1: rows touched by the
    last batch score 1 and everything else has aged to 0."""
    for s in seeds:
        for allbits in (0, 1):
            w = tg.random_tiny(s, policy="priority", batches=6)
            w.eviction_speed = 0
            w.cache_bits = (lambda b, _w=w, _v=allbits: np.full(_w.batch(b)[0].size, _v, np.uint8))
            _, recs = run_oracle(w, mutant=mutant, want64=False)
            T = w.num_tables
            R = [set() for _ in range(T)]
            U_prev = [set() for _ in range(T)]
            for b, r in enumerate(recs):
                for t in range(T):
                    P = set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                    cap = w.tables[t].cap
                    if allbits:
                        order = sorted(U_prev[t], reverse=True) + sorted((R[t] | P) - U_prev[t], reverse=True)
                    else:
                        order = sorted(R[t] | U_prev[t] | P, reverse=True)
                    R[t] = set(order[:cap])
                    assert r["resident"][t].tolist() == sorted(R[t]), f"seed {s} bits {allbits} batch {b} table {t}"
                for t, (a, e) in enumerate(segments(w, r["off"])):
                    U_prev[t] = set(r["idx"][a:e].tolist())


def pin_invariants(mutant=0, seeds=range(40)):
    for s in seeds:
        w = tg.random_tiny(s, batches=6, policy=("lru", "priority", "lfu")[s % 3])
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        prev = [0] * w.num_tables
        hpf, adm = [0] * w.num_tables, [0] * w.num_tables
        for r in recs:
            for t, (a, e) in enumerate(segments(w, r["off"])):
                f, p = r["fwd"][t], r["place"][t]
                assert f["lookups"] == e - a
                assert f["unique"] == np.unique(r["idx"][a:e]).size
                assert f["hits"] + f["misses"] == f["unique"]
                assert 0 <= f["hits_prefetch"] <= f["hits"]
                # a flag is set by one admission and ended by the row's first access
                adm[t] += p["prefetch_fill"] + p["admitted_miss"]
                hpf[t] += f["hits_prefetch"]
                assert hpf[t] <= adm[t]
                cap = w.tables[t].cap
                assert p["resident"] <= cap and p["resident"] == r["resident"][t].size
                assert p["resident"] == prev[t] - p["evicted"] + p["admitted_miss"] + p["prefetch_fill"]
                assert p["prefetch_bytes"] == p["prefetch_fill"] * w.tables[t].row_bytes
                assert f["ondemand_bytes"] == f["misses"] * w.tables[t].row_bytes
                dig = sum(splitmix64_mix_py((t << 40) | int(x)) for x in r["resident"][t]) & ((1 << 64) - 1)
                assert p["digest"] == dig
                prev[t] = p["resident"]


def pin_prefetch_quality(mutant=0, seeds=range(30)):
    """Sec. IV's coverage (Eq. coverage) counts unique vectors: brute force of
    |set(P_b) ∩ set(I_b)| and |set(P_b)| on tiny traces; exact lookahead covers
    every distinct row; a forward with no placement before it covers nothing."""
    for s in seeds:
        w = tg.random_tiny(s, batches=5, policy=("lru", "priority")[s % 2])
        if s % 3 == 0:
            w.prefetch = ("exact",)
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        for b, r in enumerate(recs):
            for t, (a, e) in enumerate(segments(w, r["off"])):
                P = set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                U = set(r["idx"][a:e].tolist())
                assert r["place"][t]["prefetch_distinct"] == len(P), f"seed {s} batch {b} table {t}"
                assert r["fwd"][t]["prefetch_covered"] == len(P & U), f"seed {s} batch {b} table {t}"
                if s % 3 == 0 and b + 1 < len(recs):
                    # exact lookahead: P_{b+1} = U_{b+1}
                    nxt = recs[b + 1]
                    a2, e2 = w.table_segment(nxt["off"], t)
                    assert nxt["fwd"][t]["prefetch_covered"] == np.unique(nxt["idx"][a2:e2]).size
    # a second forward with no placement in between covers nothing
    w = tg.random_tiny(7, batches=3)
    tabs = [w.table_values(t) for t in range(w.num_tables)]
    o = oracle.for_workload(w, tabs, mutant=mutant)
    P, poff = w.prefetch_list(0)
    assert o.placement(P, poff, None) == 0
    idx, off = w.batch(0)
    for rep in range(2):
        assert o.forward(idx, off, w.bags)[0] == 0
        for t in range(w.num_tables):
            a, e = w.table_segment(off, t)
            want = len(set(P[poff[t]:poff[t + 1]].tolist()) & set(idx[a:e].tolist())) if rep == 0 else 0
            assert o.stats(t)["prefetch_covered"] == want
    o.close()


# ----------------------------------------------------------------------------- set-associative

def pin_sa_direct_mapped(mutant=0, seeds=range(30)):
    """W = 1: every insertion replaces the set's only row, so after a placement
    a set holds its largest row of set(P) if it has one, else its largest miss
    of the last batch, else its previous row (misses first, then prefetches,
    each ascending; Alg. 1 inserts unconditionally)."""
    for s in seeds:
        w = tg.random_tiny(s, max_rows=24, max_cap=8, batches=6, policy=("lru", "priority", "lfu")[s % 3])
        w.ways = 1
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        T = w.num_tables
        held = [dict() for _ in range(T)]  # set -> row
        M_prev = [set() for _ in range(T)]
        for b, r in enumerate(recs):
            for t in range(T):
                S = min(w.tables[t].cap, w.tables[t].rows)
                P = set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                if S > 0:
                    for st in range(S):
                        ps = [x for x in P if x % S == st]
                        ms = [x for x in M_prev[t] if x % S == st]
                        if ps:
                            held[t][st] = max(ps)
                        elif ms:
                            held[t][st] = max(ms)
                assert r["resident"][t].tolist() == sorted(held[t].values()), f"seed {s} batch {b} table {t}"
            for t, (a, e) in enumerate(segments(w, r["off"])):
                U = set(r["idx"][a:e].tolist())
                R = set(held[t].values())
                M_prev[t] = U - R
                assert r["fwd"][t]["misses"] == len(U - R) and r["fwd"][t]["hits"] == len(U & R)


def pin_sa_lru_distinct_events(mutant=0, seeds=range(30)):
    """LRU_BATCH in W-way sets when every batch touches at most one row per set
    and the placement before it prefetches at most one row per set, in sets the
    batch does not touch (a prefetch before forward p and an access in forward
    p carry the same stamp p): stamps within a set never tie, and the cache
    keeps, per set, the W rows whose latest event is most recent."""
    for s in seeds:
        g = np.random.Generator(np.random.Philox(np.random.SeedSequence(4242, spawn_key=(s,))))
        S = int(g.integers(1, 5))
        W = int(g.integers(1, 4))
        per = int(g.integers(W + 1, W + 5))  # rows per set
        n = S * per
        cap = S * W + int(g.integers(0, W))  # leftover slots stay unused
        tab = np.arange(n, dtype=np.float32)[:, None]
        o = oracle.Oracle([tab], ["f32"], [cap], policy="lru", ways=W, mutant=mutant)
        last = {}
        for b in range(8):
            sets = [x for x in range(S) if g.random() < 0.7]
            P = np.array([x + S * int(g.integers(0, per)) for x in range(S) if x not in sets and g.random() < 0.6],
                         np.int32)
            assert o.placement(P, np.array([0, P.size], np.int64), None) == 0
            for x in P.tolist():
                last[x] = b
            R = set()
            for st in range(S):
                rows = sorted((x for x in last if x % S == st), key=lambda x: last[x], reverse=True)
                R |= set(rows[:W])
            assert o.resident(0).tolist() == sorted(R), f"seed {s} placement {b}"
            idx = np.array([x + S * int(g.integers(0, per)) for x in sets], np.int32)
            assert o.forward(idx, np.array([0, idx.size], np.int64), 1)[0] == 0
            st = o.stats(0)
            U = set(idx.tolist())
            assert st["hits"] == len(U & R) and st["misses"] == len(U - R)
            for x in U:
                last[x] = b
        o.close()


def pin_sa_no_eviction(mutant=0, seeds=range(12)):
    """Cap = N with W dividing N: each of the N / W sets owns exactly W rows, so
    no set overflows; the cache holds every row offered so far."""
    for s in seeds:
        w = tg.random_tiny(s, max_rows=12, batches=5)
        for tb in w.tables:
            tb.rows = 12
            tb.cap = 12
        w.ways = (1, 2, 3, 4, 6, 12)[s % 6]
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        seen = [set() for _ in w.tables]
        for b, r in enumerate(recs):
            for t in range(w.num_tables):
                seen[t] |= set(r["P"][r["poff"][t]:r["poff"][t + 1]].tolist())
                assert r["resident"][t].tolist() == sorted(seen[t]), f"seed {s} batch {b} table {t}"
                assert r["place"][t]["evicted"] == 0
            for t, (a, e) in enumerate(segments(w, r["off"])):
                U = set(r["idx"][a:e].tolist())
                assert r["fwd"][t]["misses"] == len(U - seen[t])
                seen[t] |= U


def pin_sa_invariants(mutant=0, seeds=range(30)):
    for s in seeds:
        w = tg.random_tiny(s, max_rows=30, max_cap=12, batches=6, policy=("lru", "priority", "lfu")[s % 3])
        w.ways = 1 + s % 4
        _, recs = run_oracle(w, mutant=mutant, want64=False)
        prev = [0] * w.num_tables
        hpf, adm = [0] * w.num_tables, [0] * w.num_tables
        for r in recs:
            for t, (a, e) in enumerate(segments(w, r["off"])):
                f, p = r["fwd"][t], r["place"][t]
                adm[t] += p["prefetch_fill"] + p["admitted_miss"]
                hpf[t] += f["hits_prefetch"]
                assert hpf[t] <= adm[t]
                S = min(w.tables[t].cap, w.tables[t].rows) // w.ways
                res = r["resident"][t]
                assert f["hits"] + f["misses"] == f["unique"] == np.unique(r["idx"][a:e]).size
                assert p["resident"] == res.size <= S * w.ways
                if S:
                    assert np.bincount(res % S, minlength=S).max(initial=0) <= w.ways
                else:
                    assert res.size == 0
                assert p["resident"] <= prev[t] - p["evicted"] + p["admitted_miss"] + p["prefetch_fill"]
                dig = sum(splitmix64_mix_py((t << 40) | int(x)) for x in res) & ((1 << 64) - 1)
                assert p["digest"] == dig
                prev[t] = p["resident"]


ALL_PINS = (pin_hand_examples, pin_embedding_bag, pin_splitmix, pin_lru_history, pin_lfu_history,
            pin_unbounded_cache,
            pin_zero_capacity, pin_priority_es0, pin_invariants, pin_prefetch_quality, pin_sa_direct_mapped,
            pin_sa_lru_distinct_events, pin_sa_no_eviction, pin_sa_invariants)
