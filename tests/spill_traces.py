"""Seeded churn traces that leave thousands of blocks free at once in one pool.

They drive a pool past the replay kernel's LDS table and through the paged free-block sets:
the live count rises to a peak, falls back almost to zero and rises again, so pages split,
merge, even out with neighbours and empty; random sizes make blocks split and coalesce.
Format only: event words, no allocator logic."""
from __future__ import annotations

import numpy as np

FREE_BIT = np.uint64(1 << 63)


def churn(seed: int, n_events: int, peak_live: int, lo_bytes: int, hi_bytes: int, waves: int = 2) -> np.ndarray:
    """One trace: allocations of log-uniform sizes in [lo_bytes, hi_bytes] and frees of random
    live blocks, with the live count following `waves` rise-and-fall cycles up to peak_live."""
    rng = np.random.default_rng(seed)
    out = np.empty(n_events, dtype=np.uint64)
    live = []  # alloc indices
    lo, hi = np.log(lo_bytes), np.log(hi_bytes)
    for e in range(n_events):
        phase = (e * waves / n_events) % 1.0
        target = peak_live * (1.0 - abs(2.0 * phase - 1.0))  # triangle wave 0 -> peak -> 0
        p_alloc = 0.75 if len(live) < target else 0.25
        if not live or rng.random() < p_alloc:
            out[e] = np.uint64(int(np.exp(rng.uniform(lo, hi))))
            live.append(e)
        else:
            k = int(rng.integers(len(live)))
            live[k], live[-1] = live[-1], live[k]
            out[e] = FREE_BIT | np.uint64(live.pop())
    return out


def batch(traces):
    off = np.zeros(len(traces) + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in traces])
    ev = np.concatenate(traces).astype(np.uint64) if traces else np.zeros(0, np.uint64)
    return ev, off


def fragment(seed: int, n_blocks: int, n_churn: int, lo_bytes: int = 512, hi_bytes: int = 64 << 10) -> np.ndarray:
    """One trace: n_blocks allocations, every second one freed (about n_blocks / 2 free blocks
    that cannot coalesce), n_churn random allocations and frees that reuse the holes, then every
    remaining block freed in random order (the free set coalesces back into whole segments)."""
    rng = np.random.default_rng(seed)
    lo, hi = np.log(lo_bytes), np.log(hi_bytes)
    ev = [int(np.exp(rng.uniform(lo, hi))) for _ in range(n_blocks)]
    live = list(range(0, n_blocks, 2))
    holes = list(range(1, n_blocks, 2))
    rng.shuffle(holes)
    ev += [(1 << 63) | h for h in holes]
    for _ in range(n_churn):
        if not live or rng.random() < 0.5:
            live.append(len(ev))
            ev.append(int(np.exp(rng.uniform(lo, hi))))
        else:
            k = int(rng.integers(len(live)))
            live[k], live[-1] = live[-1], live[k]
            ev.append((1 << 63) | live.pop())
    rng.shuffle(live)
    ev += [(1 << 63) | h for h in live]
    return np.array(ev, dtype=np.uint64)
