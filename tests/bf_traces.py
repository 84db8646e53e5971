"""Enumeration of tiny valid traces (format only, no allocator logic).

Every trace of at most `max_blocks` allocations in which each allocation is
freed at most once after it was made (blocks left live are persistent), over a
boundary alphabet of request sizes.  Used by the brute-force pins on the CPU
and, as one batch, by the GPU parity tests.
"""
from __future__ import annotations

import itertools

import numpy as np

from evw import A, F, KiB, MiB

# request sizes around every threshold of the paper-default parameters
ALPHABET = [0, 1, 512, 513, 256 * KiB, MiB - 1, MiB, MiB + 1, 3 * MiB, 10 * MiB - 1, 10 * MiB, 13 * MiB, 19 * MiB]


def shapes(max_blocks: int):
    """All event shapes: tuples of ('a', block) / ('f', block), allocations in block order."""
    out = []

    def rec(seq, n_alloc, live):
        out.append(tuple(seq))
        if n_alloc < max_blocks:
            rec(seq + [("a", n_alloc)], n_alloc + 1, live + [n_alloc])
        for b in live:
            rec(seq + [("f", b)], n_alloc, [x for x in live if x != b])

    rec([], 0, [])
    return [s for s in out if s]


def realise(shape, sizes):
    """Turn a shape and one size per block into event words."""
    where, ev = {}, []
    for kind, b in shape:
        if kind == "a":
            where[b] = len(ev)
            ev.append(A(sizes[b]))
        else:
            ev.append(F(where[b]))
    return ev


def enumerate_traces(max_blocks: int, alphabet=ALPHABET, sample: int | None = None, seed: int = 0):
    """All (or a seeded sample of) traces; returns a list of event-word lists."""
    traces = []
    for shp in shapes(max_blocks):
        k = sum(1 for kind, _ in shp if kind == "a")
        for sizes in itertools.product(alphabet, repeat=k):
            traces.append(realise(shp, sizes))
    if sample is not None and sample < len(traces):
        rng = np.random.default_rng(seed)
        idx = np.sort(rng.choice(len(traces), size=sample, replace=False))
        traces = [traces[i] for i in idx]
    return traces


def to_csr(traces):
    off = np.zeros(len(traces) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(t) for t in traces])
    ev = np.fromiter((w for t in traces for w in t), dtype=np.uint64, count=int(off[-1]))
    return ev, off
