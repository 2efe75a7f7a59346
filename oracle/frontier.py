"""Frontier sampling oracle (test infrastructure only).

Plain, sequential Python following Section 4.1 (Algorithm 2) for what is
sampled and Section 4.2 (Algorithms 3 and 4) for how the frontier node to
pop is chosen: a Dashboard of pins, each naming the tile of a frontier node,
probed uniformly until a pin is hit; popping clears the node's pins, adding
appends pins; when the free slots at the end are too few the live tiles are
compacted to the front, and a node that still does not fit gets the free
slots only.  V_s is the initial frontier plus every node entering the
frontier; `clip` > 1 then drops |V_s| mod clip nodes chosen uniformly
(Section 6.2's node clipping).

Random numbers: SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014), whose k-th output from state
s is mix(s + (k + 1) * 0x9E3779B97F4A7C15); stream start states are outputs
4 * id + purpose of the generator started at the seed (0 initial frontier,
1 probes, 2 neighbour choice, 3 clipping); an integer below K is
floor(r * K / 2^64).  The GPU library's host sampler is a separate
implementation of the same definition.
"""
from __future__ import annotations

import math

import numpy as np

M64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def splitmix_output(state: int, k: int) -> int:
    """The k-th (k >= 0) output of a SplitMix64 generator started at state."""
    return _mix((state + (k + 1) * GOLDEN) & M64)


class Stream:
    def __init__(self, seed: int, sub_id: int, purpose: int):
        self.state = splitmix_output(seed & M64, 4 * sub_id + purpose)
        self.count = 0

    def next(self) -> int:
        r = splitmix_output(self.state, self.count)
        self.count += 1
        return r

    def below(self, k: int) -> int:
        return (self.next() * k) >> 64


def frontier_sample(full, m: int, budget: int, eta: float, seed: int, sub_id: int,
                    clip: int = 0, trace=None) -> np.ndarray:
    """Node set of subgraph `sub_id`, sorted (int32).  trace, if a list,
    receives ("init", initial frontier) and then (popped node, new node)
    per frontier update."""
    n = int(full.n)
    indptr, indices = full.indptr, full.indices
    if n == 0:
        return np.zeros(0, np.int32)
    assert m >= 1 and budget >= m and eta >= 1.0

    def deg(v):
        return int(indptr[v + 1] - indptr[v])

    s_init, s_probe = Stream(seed, sub_id, 0), Stream(seed, sub_id, 1)
    s_nbr, s_clip = Stream(seed, sub_id, 2), Stream(seed, sub_id, 3)
    d = float(indptr[n]) / n                  # Algorithm 3: d = |E| / |V|
    cap = max(1, math.ceil(eta * m * d))      # eta * m * d slots
    db = np.full(cap, -1, np.int64)           # pins: tile number or NULL (-1)
    tiles = []                                # [node, first pin, pins, live]
    used = 0
    live_pins = 0                             # pins of frontier nodes

    def add(v, pins):
        nonlocal used, live_pins
        db[used:used + pins] = len(tiles)
        tiles.append([v, used, pins, True])
        used += pins
        live_pins += pins

    # initial frontier: m distinct nodes chosen uniformly
    mm = min(m, n)
    fs = []
    while len(fs) < mm:
        u = s_init.below(n)
        if u not in fs:
            fs.append(u)
    for v in fs:
        add(v, min(deg(v), cap - used))
    if trace is not None:
        trace.append(("init", list(fs)))
    vs = set(fs)
    for _ in range(budget - mm):
        if live_pins == 0:
            break
        # pop: probe until a pin is hit, clear that node's pins
        while True:
            t = db[s_probe.below(cap)]
            if t >= 0:
                break
        tile = tiles[t]
        v_pop = tile[0]
        db[tile[1]:tile[1] + tile[2]] = -1
        tile[3] = False
        live_pins -= tile[2]
        # a neighbour of the popped node, uniformly
        v_new = int(indices[indptr[v_pop] + s_nbr.below(deg(v_pop))])
        k = deg(v_new)
        if k > cap - used:
            # cleanup: live tiles to the front, in order
            live = [tl for tl in tiles if tl[3]]
            db[:] = -1
            tiles.clear()
            used = live_pins = 0
            for tl in live:
                add(tl[0], tl[2])
        add(v_new, min(k, cap - used))
        vs.add(v_new)
        if trace is not None:
            trace.append((v_pop, v_new))
    out = sorted(vs)
    if clip > 1:
        for _ in range(len(out) % clip):
            del out[s_clip.below(len(out))]
    return np.array(out, np.int32)
