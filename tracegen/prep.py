"""Seeded synthetic profiler streams for the trace-preparation steps (Sections 3.2, 3.3).

A stand-in for the PyTorch-profiler traces the paper consumes: the allocator instant events
(timestamp, address, +/- bytes) of a CPU training run, one category per allocation (the role
the Analyzer's operator attribution would give it), and the user-annotation timestamps of
`profiler.step()` (iteration starts) and `optimizer.zero_grad()`.

The modelled loop: parameters allocated once (model.to(device)); per iteration a batch of
input and label tensors, a forward pass with one activation per layer and random short-lived
temporaries, a loss, a backward pass that creates one gradient per parameter tensor and frees
the activations in reverse, and an Adam step whose two state tensors per parameter are
allocated in the first iteration only.  `zero_grad` runs at the iteration start (POS1) or just
before the backward pass (POS0), the two placements of the paper's Fig. 1.  The CPU lifetimes
are deliberately not the GPU ones: batches are never freed, gradients are freed right after
the optimizer step, and most parameters are freed at the very end.  Addresses come from a
reuse-first address pool, so the same address is reused by later blocks.

Format only: no allocator or orchestration logic lives here.
"""
from __future__ import annotations

import numpy as np

RAW_DTYPE = np.dtype([("ts", np.int64), ("addr", np.uint64), ("bytes", np.int64)])
CAT_OTHER, CAT_PARAMETER, CAT_BATCH, CAT_GRADIENT, CAT_OPTIMIZER = 0, 1, 2, 3, 4


class _Stream:
    def __init__(self, rng, cap):
        self.rng = rng
        self.cap = cap
        self.ts = np.empty(cap, np.int64)
        self.addr = np.empty(cap, np.uint64)
        self.nb = np.empty(cap, np.int64)
        self.cat = np.empty(cap, np.int32)
        self.n = 0
        self.t = int(rng.integers(0, 1000))
        self.pool = []          # addresses free for reuse
        self.bump = 0x7F0000000000

    def full(self):
        return self.n >= self.cap

    def tick(self):
        self.t += int(self.rng.integers(1, 64))
        return self.t

    def _push(self, a, nb, cat):
        if self.n < self.cap:
            self.ts[self.n], self.addr[self.n], self.nb[self.n], self.cat[self.n] = self.tick(), a, nb, cat
            self.n += 1

    def alloc(self, nbytes, cat):
        if self.pool and self.rng.random() < 0.85:
            a = self.pool.pop(int(self.rng.integers(len(self.pool))) if self.rng.random() < 0.3 else -1)
        else:
            a = self.bump
            self.bump += (int(nbytes) + 511) // 512 * 512
        self._push(a, int(nbytes), cat)
        return a, int(nbytes)

    def free(self, blk):
        a, nbytes = blk
        self._push(a, -nbytes, CAT_OTHER)
        self.pool.append(a)


def training_profile(seed: int, n_events: int, layers: int = 24, batch: int = 8, pos: str = "POS1",
                     temp_p: float = 0.5):
    """One trace of exactly n_events raw events (the loop is cut where the budget ends).
    Returns (raw[RAW_DTYPE], category int32[], step_ts int64[], zero_grad_ts int64[])."""
    rng = np.random.default_rng(seed)
    s = _Stream(rng, n_events)
    w_size = [int(np.exp(rng.uniform(np.log(64 << 10), np.log(64 << 20)))) // 4 * 4 for _ in range(layers)]
    b_size = [int(rng.integers(1, 4096)) * 4 for _ in range(layers)]
    act = [batch * int(np.exp(rng.uniform(np.log(16 << 10), np.log(4 << 20)))) // 4 * 4 for _ in range(layers)]
    params = [s.alloc(w_size[l], CAT_PARAMETER) for l in range(layers)] + \
             [s.alloc(b_size[l], CAT_PARAMETER) for l in range(layers)]
    steps, zgs = [], []
    it = 0
    while not s.full():
        steps.append(s.tick())
        if pos == "POS1":
            zgs.append(s.tick())
        x = s.alloc(batch * 3 * 224 * 224 * 4 // 16, CAT_BATCH)
        y = s.alloc(batch * 8, CAT_BATCH)
        del x, y  # the CPU trace never frees the batch
        acts = []
        for l in range(layers):
            acts.append(s.alloc(act[l], CAT_OTHER))
            if rng.random() < temp_p:
                s.free(s.alloc(int(np.exp(rng.uniform(np.log(512), np.log(max(act[l], 1024))))), CAT_OTHER))
        loss = s.alloc(4 * batch, CAT_OTHER)
        if pos == "POS0":
            zgs.append(s.tick())
        grads = []
        for l in reversed(range(layers)):
            grads.append(s.alloc(w_size[l], CAT_GRADIENT))
            grads.append(s.alloc(b_size[l], CAT_GRADIENT))
            s.free(acts[l])
            if rng.random() < temp_p:
                s.free(s.alloc(int(np.exp(rng.uniform(np.log(512), np.log(max(act[l], 1024))))), CAT_OTHER))
        s.free(loss)
        if it == 0:
            for l in range(layers):
                for size in (w_size[l], b_size[l]):
                    s.alloc(size, CAT_OPTIMIZER)
                    s.alloc(size, CAT_OPTIMIZER)
        for g in grads:  # the CPU frees gradients right after the step
            s.free(g)
        it += 1
    for p_ in params[: (3 * len(params)) // 4]:
        s.free(p_)
    raw = np.zeros(s.n, RAW_DTYPE)
    raw["ts"], raw["addr"], raw["bytes"] = s.ts[: s.n], s.addr[: s.n], s.nb[: s.n]
    return raw, s.cat[: s.n].copy(), np.array(steps, np.int64), np.array(zgs, np.int64)


def batch_profiles(n_traces: int, n_events: int, seed: int = 0, pos: str = "POS1", layers: int = 24):
    """CSR batch: trace t uses seed (seed << 20) + t and batch size 1 + t % 16.
    Returns (raw, category, raw_off, steps, step_off, zero_grads, zg_off)."""
    parts = [training_profile((seed << 20) + t, n_events, layers=layers, batch=1 + t % 16, pos=pos)
             for t in range(n_traces)]

    def csr(arrs, dtype):
        off = np.zeros(len(arrs) + 1, np.int64)
        off[1:] = np.cumsum([len(a) for a in arrs])
        return (np.concatenate(arrs).astype(dtype) if arrs else np.zeros(0, dtype)), off

    raw, roff = csr([p[0] for p in parts], RAW_DTYPE)
    cat, _ = csr([p[1] for p in parts], np.int32)
    st, soff = csr([p[2] for p in parts], np.int64)
    zg, zoff = csr([p[3] for p in parts], np.int64)
    return raw, cat, roff, st, soff, zg, zoff
