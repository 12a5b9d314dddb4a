"""A host model of the attention merge's counter protocol (one 64-bit word per row set), run over random
schedules of the pieces' starts and arrivals, with the field layout read from the kernels' header.

Each piece adds (1, its XCD id, the id's square) to the word when it starts and keeps the value before its
add; when its rows are stored it adds an arrival and its bit.  A piece whose arrival finds the whole set
started waits for every arrival (or for the word's reset to zero) and merges its own slice; the piece whose
start completed the set also merges the slices of the pieces that had arrived before that; the last arrival
resets the word.  The model checks, for every schedule: each slice is merged exactly once, every wait is for
pieces that have started (so it ends), the word ends at zero, and a merging piece flags the set exactly when
its pieces did not all run on one XCD.
"""
import os
import re

import numpy as np
import pytest

HEADER = os.path.join(os.path.dirname(__file__), "..", "paper_2606_00535_amd", "csrc", "kernels.h")


def fields():
    text = open(HEADER).read()
    m = re.search(r"constexpr int kCtrCountBits = (\d+), kCtrArrived = (\d+), kCtrMask = (\d+), "
                  r"kCtrXcdSum = (\d+), kCtrXcdSq = (\d+);", text)
    assert m, "counter field constants not found"
    max_splits = int(re.search(r"constexpr int kAttnMaxSplits = (\d+);", text).group(1))
    return tuple(int(x) for x in m.groups()) + (max_splits,)


CB, ARR, MASK, XSUM, XSQ, MAXS = fields()
CNT = (1 << CB) - 1
M64 = (1 << 64) - 1


def run_schedule(S, xcds, rng):
    """One random interleaving of S pieces; returns (slices merged per piece, flags, final word)."""
    word = 0
    start_old = [None] * S
    state = ["new"] * S          # new -> started -> waiting/done
    merged = [0] * S
    flagged = [False] * S
    waiting = {}                 # piece -> bool (coop, still waiting)
    coop_of = [False] * S
    while True:
        # a waiting piece may finish once its condition holds
        ready = [k for k in waiting if ((word >> ARR) & CNT) == S or (word & CNT) == 0]
        movable = [k for k in range(S) if state[k] in ("new", "started")] + ready
        if not movable:
            break
        k = movable[rng.integers(len(movable))]
        if k in waiting:                         # the wait ends
            del waiting[k]
            state[k] = "done"
            continue
        if state[k] == "new":                    # start
            x = xcds[k]
            start_old[k] = word
            word = (word + (1 | (x << XSUM) | ((x * x) << XSQ))) & M64
            state[k] = "started"
            continue
        # arrival
        old = word
        word = (word + ((1 << ARR) | (1 << (MASK + k)))) & M64
        coop = (old & CNT) == S
        last = ((old >> ARR) & CNT) == S - 1
        coop_of[k] = coop
        if coop:
            x = xcds[k]
            ssum = (old >> XSUM) & ((1 << (XSQ - XSUM)) - 1)
            ssq = old >> XSQ
            flagged[k] = ssum != S * x or ssq != S * x * x
            # every piece this one would wait for has started (the set is complete)
            assert (old & CNT) == S
        slices = (1 << k) if coop else 0
        if (start_old[k] & CNT) == S - 1:
            slices |= (start_old[k] >> MASK) & ((1 << S) - 1)
        merged[k] = slices
        if last:
            word = 0
            state[k] = "done"
        elif coop:
            waiting[k] = True
            state[k] = "waiting"
        else:
            state[k] = "done"
    assert not waiting, "a wait never ended"
    assert all(st == "done" for st in state)
    return merged, flagged, coop_of, word


@pytest.mark.parametrize("S", [2, 3, 5, 8, 17, 32])
def test_every_slice_merged_once_and_word_cleared(S):
    assert S <= MAXS
    rng = np.random.default_rng(S)
    for _ in range(300):
        merged, flagged, coop_of, word = run_schedule(S, [3] * S, rng)
        assert all(coop_of[k] for k in range(S) if merged[k]), "a merger that had not seen the whole set start"
        total = 0
        for m in merged:
            assert total & m == 0, "a slice merged twice"
            total |= m
        assert total == (1 << S) - 1, "a slice never merged"
        assert word == 0
        assert not any(flagged)


@pytest.mark.parametrize("S", [2, 4, 8, 32])
def test_split_xcd_is_flagged_by_every_merger(S):
    rng = np.random.default_rng(100 + S)
    for _ in range(300):
        xcds = [int(v) for v in rng.integers(0, 8, S)]
        if len(set(xcds)) == 1:
            xcds[0] = (xcds[0] + 1) % 8
        merged, flagged, coop_of, word = run_schedule(S, xcds, rng)
        mergers = [k for k in range(S) if merged[k]]
        assert mergers and all(coop_of[k] and flagged[k] for k in mergers)
        assert word == 0


def test_field_widths_hold_the_largest_set():
    # counts up to kAttnMaxSplits, the arrival mask, and sums of squares of ids up to 7 all fit their fields
    assert MAXS <= CNT and ARR >= CB and MASK >= ARR + CB and XSUM >= MASK + MAXS
    assert MAXS * 7 < (1 << (XSQ - XSUM)) and MAXS * 49 < (1 << (64 - XSQ))
    # sum S x and sum of squares S x^2 force equal ids: a pair (x, y) with the same sums does not exist
    for S in (2, 3, 8, 32):
        for x in range(8):
            for y in range(8):
                if x != y:
                    ids = [x] * (S - 1) + [y]
                    assert not (sum(ids) == S * x and sum(i * i for i in ids) == S * x * x)
