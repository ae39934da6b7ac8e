"""Pins of the SSD -> DRAM tier oracle (oracle/preload.py) against what the
passage and combinatorics fix: the decisions reach the minimum number of
layer loads that any choice of victims can reach (exhaustive search on small
stacks), every layer is in DRAM when it is used, the fixed area is never
loaded or evicted, and a dynamic area that holds every dynamic layer loads
each of them once."""
import functools
import sys

import pytest

from oracle.preload import TwoLevelDram


def _min_loads(L, fixed, slots, a, tokens):
    """Fewest loads over every legal sequence of victim choices (dynamic
    programming over (position, slot contents)): the window W(l) is made
    resident in order, a victim may be any slot whose layer is outside W(l),
    the layer in use must be loaded, a look-ahead load may be skipped only if
    no slot can be given up."""
    seq = [l for _ in range(tokens) for l in range(L)]
    sys.setrecursionlimit(10000)

    @functools.lru_cache(None)
    def best(pos, state):
        if pos == len(seq):
            return 0
        l = seq[pos]
        window = [(l + j) % L for j in range(a + 1)]

        def rec(i, st):
            if i == len(window):
                return best(pos + 1, st)
            m = window[i]
            if m < fixed or m in st:
                return rec(i + 1, st)
            empty = [s for s, v in enumerate(st) if v < 0]
            if empty:
                st2 = list(st)
                st2[empty[0]] = m
                return 1 + rec(i + 1, tuple(st2))
            cand = [s for s, v in enumerate(st) if v not in window]
            if not cand:
                return 10 ** 9 if m == l else rec(i + 1, st)
            res = 10 ** 9
            for s in cand:
                st2 = list(st)
                st2[s] = m
                res = min(res, 1 + rec(i + 1, tuple(st2)))
            return res

        return rec(0, state)

    return best(0, tuple([-1] * slots))


CASES = [(L, fixed, slots, a) for L in range(3, 8) for fixed in range(0, L) for a in (1, 2)
         for slots in range(a + 1, L - fixed + 1)]


@pytest.mark.parametrize("L,fixed,slots,a", CASES)
def test_loads_are_minimal(L, fixed, slots, a):
    c = TwoLevelDram(L, fixed, slots, a)
    c.run_tokens(3)
    assert len(c.log) == _min_loads(L, fixed, slots, a, 3)


@pytest.mark.parametrize("L,fixed,slots,a", [(12, 3, 4, 2), (10, 0, 3, 2), (9, 2, 7, 1),
                                             (16, 4, 6, 3), (8, 8, 2, 1)])
def test_invariants(L, fixed, slots, a):
    c = TwoLevelDram(L, fixed, slots, a)
    seq = [l for _ in range(5) for l in range(L)]
    loaded = []
    for pos, l in enumerate(seq):
        before = len(c.log)
        c.use(l)
        window = {(l + j) % L for j in range(a + 1)}
        assert c.resident(l)
        for (_, m, s, old) in c.log[before:]:
            loaded.append(m)
            assert m >= fixed and old not in window
            if old >= 0:
                # furthest next use among the slots that could be given up,
                # by scanning the use sequence forward
                def next_use(v):
                    for q in range(pos + 1, len(seq) + L):
                        if (q % L) == v:
                            return q
                    return 10 ** 9
                others = [v for v in c.slot_layer if v not in window and v != m]
                assert all(next_use(old) >= next_use(v) for v in others)
    if fixed + slots >= L:
        assert sorted(loaded) == list(range(fixed, L))  # each dynamic layer once


def test_rejects_too_few_slots():
    with pytest.raises(ValueError):
        TwoLevelDram(10, 2, 2, 2)
