"""Every planted mistake in the oracle (built on the CPU with ORACLE_MUTANT=k)
must trip at least one pin; otherwise the pins would not guard that part."""
import pytest

import oracle
import oracle_pins as op

MUTANTS = {
    1: "ties evict the higher row id",
    2: "no aging under PRIORITY",
    3: "prefetch overwrites a larger score",
    4: "last caching bit wins instead of OR",
    5: "last index of every bag dropped",
    6: "prefetch flag survives an access",
    7: "LRU prefetch scored like a touch",
    8: "digest forgets the table id",
    9: "aging does not saturate at 0",
    10: "coverage counts lookups with their repeats",
    11: "set-associative: ties evict the last way",
    12: "set-associative: the set ages before the victim is chosen",
    13: "set-associative: prefetch rows inserted before the misses",
    14: "set-associative: events of a set in descending row order",
    15: "set-associative: aging once per placement instead of per eviction",
    16: "set-associative: set index taken modulo the ways",
    17: "LFU counts every access instead of every batch",
    18: "an admitted miss that the prefetch list names is not flagged as prefetched",
}


@pytest.mark.parametrize("k", sorted(MUTANTS), ids=lambda k: f"mutant{k}")
def test_mutant_is_caught(k, tmp_path):
    oracle.build(mutant=k)
    caught = []
    for pin in op.ALL_PINS:
        try:
            pin(k)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {k} ({MUTANTS[k]}) passed every pin"
