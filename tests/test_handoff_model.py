"""CPU model of the persistent kernels' item handoff.

The attention kernels run a persistent grid of G work-groups over a work
list of n items.  Two protocols hand items out:

* forward (two ahead): work-group b starts on item b and has item 2G-1-b as
  its static second item (used only when it exists); while an item runs, it
  pops one index from a global counter (pop k -> item 2G + k) for the item
  after next; at an item's end it moves on to its next item if that index is
  below n, else it stops.
* backward (one ahead): work-group b starts on item b; each item pops
  (pop k -> item G + k) at its last step the item that follows it.

The model replays both protocols under random item durations and random
orders of simultaneous pops, and checks that every item runs exactly once
and every work-group stops (no lost, doubled or invented item, no wait on an
index that never comes).  The kernels' index arithmetic is written out here
from the protocol, not taken from the kernel source.
"""
import heapq

import numpy as np
import pytest


def run_forward(n, G, cost, rng):
    """Returns the list of items each work-group ran."""
    G = min(G, n)
    ran = [[] for _ in range(G)]
    pop = 0
    events = []                                  # (time, tiebreak, wg, phase, state)
    for b in range(G):
        state = dict(cur=b, nxt=2 * G - 1 - b, nxt2=None)
        heapq.heappush(events, (0.0, rng.random(), b, "start", state))
    while events:
        t, _, b, phase, st = heapq.heappop(events)
        if phase == "start":
            ran[b].append(st["cur"])
            c = cost[st["cur"]]
            # the pop happens one step before the item's last (at its only
            # step for one-step items); simultaneous pops are ordered randomly
            heapq.heappush(events, (t + max(c - 1, 0) + 0.5, rng.random(), b, "pop", st))
        elif phase == "pop":
            st["nxt2"] = pop + 2 * G
            pop += 1
            heapq.heappush(events, (t + 0.5 + (1 if cost[st["cur"]] > 1 else 0),
                                    rng.random(), b, "end", st))
        else:                                    # end of the item
            if st["nxt"] >= n:
                continue                         # has_next is false: stop
            nst = dict(cur=st["nxt"], nxt=st["nxt2"], nxt2=None)
            heapq.heappush(events, (t, rng.random(), b, "start", nst))
    return ran


def run_backward(n, G, cost, rng):
    G = min(G, n)
    ran = [[] for _ in range(G)]
    pop = 0
    events = [(0.0, rng.random(), b, "start", dict(cur=b)) for b in range(G)]
    heapq.heapify(events)
    while events:
        t, _, b, phase, st = heapq.heappop(events)
        if phase == "start":
            ran[b].append(st["cur"])
            heapq.heappush(events, (t + cost[st["cur"]] - 0.5, rng.random(), b, "pop", st))
        elif phase == "pop":                     # at the item's last step
            st["nxt"] = pop + G
            pop += 1
            heapq.heappush(events, (t + 0.5, rng.random(), b, "end", st))
        else:
            if st["nxt"] < n:
                heapq.heappush(events, (t, rng.random(), b, "start", dict(cur=st["nxt"])))
    return ran


def check_once(ran, n):
    flat = [i for r in ran for i in r]
    assert sorted(flat) == list(range(n)), "an item was lost, doubled or invented"


@pytest.mark.parametrize("proto", [run_forward, run_backward])
def test_every_item_runs_once(proto):
    rng = np.random.default_rng(0)
    for trial in range(300):
        n = int(rng.integers(1, 400))
        G = int(rng.integers(1, 64))
        # longest-first costs (the scheduler's order), with ties and 1-step items
        cost = np.sort(rng.integers(1, 9, size=n))[::-1]
        ran = proto(n, G, cost, rng)
        check_once(ran, n)


@pytest.mark.parametrize("proto", [run_forward, run_backward])
def test_small_lists_and_wide_grids(proto):
    rng = np.random.default_rng(1)
    for n in range(1, 12):
        for G in range(1, 2 * n + 3):
            for _ in range(5):
                cost = rng.integers(1, 4, size=n)
                check_once(proto(n, G, cost, rng), n)
