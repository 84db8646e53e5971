"""Event-word spelling for hand-written traces (format only, no allocator logic)."""
FREE_BIT = 1 << 63
KiB, MiB = 1 << 10, 1 << 20


def A(nbytes: int) -> int:
    """ALLOC word for a request of nbytes."""
    return int(nbytes)


def F(alloc_index: int) -> int:
    """FREE word releasing the allocation made by event alloc_index of the same trace."""
    return FREE_BIT | int(alloc_index)
