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


def spill_mix(seed: int, n_frag: int = 2400, iters: int = 30, large: bool = False) -> np.ndarray:
    """One trace whose small pool passes 768 free blocks early, with short-lived temporaries
    (freed 1 to 150 events after their allocation) all around that point: a block live until
    the fragmentation is over (so that a chunked replay's first chunk holds all of it), n_frag
    1 KiB blocks, every other one freed, the rest freed, then `iters` balanced iterations (clean
    positions for later chunks).  A random lead of temporaries moves the point within its
    64-event tile.  large: the blocks and temporaries are of the large pool (just over 1 MiB)."""
    rng = np.random.default_rng(seed)
    ev: list[int] = []
    due: list[tuple[int, int]] = []  # (event index at which to free, allocation index)

    def put(word: int) -> None:
        ev.append(word)
        while True:  # the temporaries whose time has come, in order
            ready = [x for x in due if x[0] <= len(ev)]
            if not ready:
                return
            x = min(ready)
            due.remove(x)
            ev.append((1 << 63) | x[1])

    def temp() -> None:
        a = len(ev)
        due.append((a + 1 + int(rng.integers(1, 150)), a))
        k = int(rng.integers(1, 8))
        put((1 << 20) + k * 8192 if large else k * 128)

    put(64)  # live until the fragmentation is over: no clean position before it (the first chunk)
    for _ in range(int(rng.integers(0, 200))):
        temp()
    blocks = []
    for _ in range(n_frag):
        blocks.append(len(ev))
        put((1 << 20) + 4096 if large else 1024)
        if rng.random() < 0.3:
            temp()
    for j in list(range(0, n_frag, 2)) + list(range(1, n_frag, 2)):
        put((1 << 63) | blocks[j])
        if rng.random() < 0.5:
            temp()
    for x in sorted(due):
        ev.append((1 << 63) | x[1])
    due.clear()
    ev.append((1 << 63) | 0)
    for _ in range(iters):
        s0 = len(ev)
        m = int(rng.integers(20, 60))
        for _ in range(m):
            ev.append(int(rng.integers(1, 64)) * 512)
        order = rng.permutation(m)
        ev += [(1 << 63) | (s0 + int(j)) for j in order]
    return np.array(ev, dtype=np.uint64)
