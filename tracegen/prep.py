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

With windows=True a trace also carries its execution windows in start order, each with its
enclosing window: components (python_function: model.to, ProfilerStep, dataloader, each layer's
forward and backward, the loss module, optimizer.step) and the operators (cpu_op) inside them,
each operator tagged with the role of the blocks it produces (parameters, batch data,
gradients); the optimizer.step() component is tagged "optimizer" to mark the phase in which the
optimizer states are found by their sizes.  About one layer in ten also
allocates a script-level temporary outside every operator window.

Format only: no allocator, attribution or orchestration logic lives here.
"""
from __future__ import annotations

import numpy as np

RAW_DTYPE = np.dtype([("ts", np.int64), ("addr", np.uint64), ("bytes", np.int64)])
WINDOW_DTYPE = np.dtype([("start", np.int64), ("end", np.int64), ("parent", np.int32), ("kind", np.int32),
                         ("category", np.int32), ("pad", np.int32)])
CAT_OTHER, CAT_PARAMETER, CAT_BATCH, CAT_GRADIENT, CAT_OPTIMIZER = 0, 1, 2, 3, 4
WIN_COMPONENT, WIN_OPERATOR = 0, 1


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
        self.win = []           # [start, end, parent, kind, category]
        self.open = []          # indices of the windows currently open (innermost last)

    def full(self):
        return self.n >= self.cap

    def enter(self, kind, category=CAT_OTHER):
        """Open an execution window (a python_function component or a cpu_op operator)."""
        self.win.append([self.tick(), -1, self.open[-1] if self.open else -1, kind, category])
        self.open.append(len(self.win) - 1)

    def leave(self):
        self.win[self.open.pop()][1] = self.tick()

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
                     temp_p: float = 0.5, windows: bool = False):
    """One trace of exactly n_events raw events (the loop is cut where the budget ends).
    Returns (raw[RAW_DTYPE], category int32[], step_ts int64[], zero_grad_ts int64[]) and, with
    windows=True, also the execution windows [WINDOW_DTYPE] ordered by start."""
    rng = np.random.default_rng(seed)
    s = _Stream(rng, n_events)
    w_size = [int(np.exp(rng.uniform(np.log(64 << 10), np.log(64 << 20)))) // 4 * 4 for _ in range(layers)]
    b_size = [int(rng.integers(1, 4096)) * 4 for _ in range(layers)]
    act = [batch * int(np.exp(rng.uniform(np.log(16 << 10), np.log(4 << 20)))) // 4 * 4 for _ in range(layers)]
    s.enter(WIN_COMPONENT)                      # model.to(device)
    s.enter(WIN_OPERATOR, CAT_PARAMETER)
    params = [s.alloc(w_size[l], CAT_PARAMETER) for l in range(layers)] + \
             [s.alloc(b_size[l], CAT_PARAMETER) for l in range(layers)]
    s.leave()
    s.leave()
    steps, zgs = [], []
    it = 0
    def temp(upper):
        return int(np.exp(rng.uniform(np.log(512), np.log(max(upper, 1024)))))

    while not s.full():
        steps.append(s.tick())
        s.enter(WIN_COMPONENT)                  # ProfilerStep#it
        if pos == "POS1":
            zgs.append(s.tick())
        s.enter(WIN_COMPONENT)                  # dataloader.__next__
        s.enter(WIN_OPERATOR, CAT_BATCH)
        x = s.alloc(batch * 3 * 224 * 224 * 4 // 16, CAT_BATCH)
        y = s.alloc(batch * 8, CAT_BATCH)
        del x, y  # the CPU trace never frees the batch
        s.leave()
        s.leave()
        acts = []
        for l in range(layers):
            s.enter(WIN_COMPONENT)              # layer l forward
            s.enter(WIN_OPERATOR)               # its compute op: the activation outlives the layer
            acts.append(s.alloc(act[l], CAT_OTHER))
            if rng.random() < temp_p:
                s.free(s.alloc(temp(act[l]), CAT_OTHER))
            s.leave()
            s.leave()
            if rng.random() < 0.1:              # a script-level temporary outside every operator
                s.free(s.alloc(temp(4096), CAT_OTHER))
        s.enter(WIN_COMPONENT)                  # the loss module
        s.enter(WIN_OPERATOR)
        loss = s.alloc(4 * batch, CAT_OTHER)
        s.leave()
        s.leave()
        if pos == "POS0":
            zgs.append(s.tick())
        grads = []
        for l in reversed(range(layers)):
            s.enter(WIN_COMPONENT)              # layer l backward
            s.enter(WIN_OPERATOR, CAT_GRADIENT)
            grads.append(s.alloc(w_size[l], CAT_GRADIENT))
            grads.append(s.alloc(b_size[l], CAT_GRADIENT))
            s.free(acts[l])
            if rng.random() < temp_p:
                s.free(s.alloc(temp(act[l]), CAT_OTHER))
            s.leave()
            s.leave()
        s.free(loss)
        s.enter(WIN_COMPONENT, CAT_OPTIMIZER)   # optimizer.step(): the phase the optimizer rule looks at
        s.enter(WIN_OPERATOR)                   # its operator gives its products no role of its own
        if it == 0:
            for l in range(layers):
                for size in (w_size[l], b_size[l]):
                    s.alloc(size, CAT_OPTIMIZER)
                    s.alloc(size, CAT_OPTIMIZER)
        if rng.random() < temp_p:
            s.free(s.alloc(temp(1 << 20), CAT_OTHER))
        s.leave()
        s.leave()
        for g in grads:  # the CPU frees gradients right after the step
            s.free(g)
        s.leave()                               # end of ProfilerStep#it
        it += 1
    for p_ in params[: (3 * len(params)) // 4]:
        s.free(p_)
    raw = np.zeros(s.n, RAW_DTYPE)
    raw["ts"], raw["addr"], raw["bytes"] = s.ts[: s.n], s.addr[: s.n], s.nb[: s.n]
    out = (raw, s.cat[: s.n].copy(), np.array(steps, np.int64), np.array(zgs, np.int64))
    if not windows:
        return out
    w = np.zeros(len(s.win), WINDOW_DTYPE)
    for i, (a, b, par, kind, cat) in enumerate(s.win):
        w[i] = (a, b if b >= 0 else s.t + 1, par, kind, cat, 0)
    return out + (w,)


def batch_profiles(n_traces: int, n_events: int, seed: int = 0, pos: str = "POS1", layers: int = 24,
                   windows: bool = False):
    """CSR batch: trace t uses seed (seed << 20) + t and batch size 1 + t % 16.
    Returns (raw, category, raw_off, steps, step_off, zero_grads, zg_off) and, with windows=True,
    also (windows, window_off)."""
    parts = [training_profile((seed << 20) + t, n_events, layers=layers, batch=1 + t % 16, pos=pos, windows=windows)
             for t in range(n_traces)]

    def csr(arrs, dtype):
        off = np.zeros(len(arrs) + 1, np.int64)
        off[1:] = np.cumsum([len(a) for a in arrs])
        return (np.concatenate(arrs).astype(dtype) if arrs else np.zeros(0, dtype)), off

    raw, roff = csr([p[0] for p in parts], RAW_DTYPE)
    cat, _ = csr([p[1] for p in parts], np.int32)
    st, soff = csr([p[2] for p in parts], np.int64)
    zg, zoff = csr([p[3] for p in parts], np.int64)
    if not windows:
        return raw, cat, roff, st, soff, zg, zoff
    win, woff = csr([p[4] for p in parts], WINDOW_DTYPE)
    return raw, cat, roff, st, soff, zg, zoff, win, woff
