"""Brute-force model of the Memory Simulator (Section 3.4), for tiny traces.

A second implementation of the same allocator reading as the oracle, written
differently on purpose so that the two pin each other:
  * each segment is a Python list of [offset, size, is_free] intervals;
  * best fit scans every interval of every segment of the pool (no index);
  * coalescing re-normalises the whole segment after each free (adjacent free
    intervals fused until none remain);
  * OOM reclaim scans all segments.
Only used on traces of a few events.  Never timed.
"""
from __future__ import annotations

MiB = 1 << 20
FREE_BIT = 1 << 63
MAX_REQUEST = 1 << 48
POOL_CREATED_LIMIT = 1 << 61
OK, OOM, BAD_FREE, BAD_EVENT, OVERFLOW = 0, 1, 2, 3, 4


def run(events, p):
    """Returns (result dict, series list)."""
    segs = []  # dicts: base, size, pool, live, iv (list of [off, size, free])
    bump = 0
    allocated = reserved = 0
    created = released = 0
    created_bytes = [0, 0]
    where = {}  # alloc event index -> (segment index, offset) or None for no-op
    req = {}
    freed = set()
    is_alloc = set()
    series = []
    res = dict(peak_allocated=0, peak_reserved=0, peak_allocated_event=-1, peak_reserved_event=-1,
               max_free_blocks_small=0, max_free_blocks_large=0, stop_event=-1, status=OK)

    def pool_of(r):
        return 0 if r <= p["small_max_bytes"] else 1

    def nfree(pool):
        return sum(1 for g in segs if g["live"] and g["pool"] == pool for iv in g["iv"] if iv[2])

    def normalise(g):
        out = []
        for iv in g["iv"]:
            if out and out[-1][2] and iv[2]:
                out[-1][1] += iv[1]
            else:
                out.append(list(iv))
        g["iv"] = out

    def idle(g):
        return g["live"] and len(g["iv"]) == 1 and g["iv"][0][2]

    status = OK
    for e, w in enumerate(events):
        w = int(w)
        if w & FREE_BIT:
            if (w >> 32) & 0x7FFFFFFF:
                status = BAD_EVENT
            else:
                h = w & 0xFFFFFFFF
                if h >= e or h not in is_alloc or h in freed:
                    status = BAD_FREE
                else:
                    freed.add(h)
                    loc = where[h]
                    if loc is not None:
                        gi, off = loc
                        g = segs[gi]
                        for iv in g["iv"]:
                            if iv[0] == off:
                                assert not iv[2]
                                iv[2] = True
                                break
                        else:
                            raise AssertionError("block not found")
                        normalise(g)
                        allocated -= req[h]
        else:
            s = w
            if s > MAX_REQUEST:
                status = BAD_EVENT
            else:
                is_alloc.add(e)
                g_ = p["round_bytes"]
                r = -(-s // g_) * g_
                if r == 0:
                    where[e] = None
                else:
                    pool = pool_of(r)
                    best = None  # (size, absolute address, seg index, interval index)
                    for gi, g in enumerate(segs):
                        if not g["live"] or g["pool"] != pool:
                            continue
                        for ii, iv in enumerate(g["iv"]):
                            if iv[2] and iv[1] >= r:
                                key = (iv[1], g["base"] + iv[0], gi, ii)
                                if best is None or key[:2] < best[:2]:
                                    best = key
                    if best is None:
                        if pool == 0:
                            S = p["small_segment_bytes"]
                        elif r < p["min_large_alloc_bytes"]:
                            S = p["mid_segment_bytes"]
                        else:
                            q = p["large_round_bytes"]
                            S = -(-r // q) * q
                        if created_bytes[pool] + S > POOL_CREATED_LIMIT:
                            status = OVERFLOW
                        else:
                            cap = p["device_capacity_bytes"]
                            if reserved + S > cap:
                                idle_bytes = sum(g["size"] for g in segs if idle(g))
                                if reserved - idle_bytes + S > cap:
                                    status = OOM
                                else:
                                    for g in segs:
                                        if idle(g):
                                            g["live"] = False
                                            reserved -= g["size"]
                                            released += 1
                            if status == OK:
                                segs.append(dict(base=bump, size=S, pool=pool, live=True, iv=[[0, S, True]]))
                                bump += S
                                reserved += S
                                created += 1
                                created_bytes[pool] += S
                                best = (S, segs[-1]["base"], len(segs) - 1, 0)
                    if status == OK:
                        _, _, gi, ii = best
                        g = segs[gi]
                        off, size, _ = g["iv"][ii]
                        rem = size - r
                        split_min = p["split_min_small_bytes"] if pool == 0 else p["split_min_large_bytes"]
                        if rem >= split_min:
                            g["iv"][ii:ii + 1] = [[off, r, False], [off + r, rem, True]]
                        else:
                            g["iv"][ii][2] = False
                        where[e] = (gi, off)
                        req[e] = r
                        allocated += r
        if status != OK:
            res["status"] = status
            res["stop_event"] = e
            series.extend([-1] * (len(events) - e))
            break
        series.append(reserved)
        if allocated > res["peak_allocated"]:
            res["peak_allocated"], res["peak_allocated_event"] = allocated, e
        if reserved > res["peak_reserved"]:
            res["peak_reserved"], res["peak_reserved_event"] = reserved, e
        res["max_free_blocks_small"] = max(res["max_free_blocks_small"], nfree(0))
        res["max_free_blocks_large"] = max(res["max_free_blocks_large"], nfree(1))
    res.update(final_allocated=allocated, final_reserved=reserved, segments_created=created,
               segments_released=released)
    return res, series
