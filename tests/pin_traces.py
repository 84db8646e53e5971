"""The hand-derived example traces (their expected values are asserted on the
oracle in test_oracle_pins.py), gathered so the GPU tests can replay them all
in one batch per parameter set."""
from evw import A, F, KiB, MiB

import oracle

P = oracle.paper_params()
PT = oracle.pytorch_like_params()


def catalogue():
    """[(name, trace, params)]"""
    cap = lambda c: oracle.paper_params(device_capacity_bytes=c)  # noqa: E731
    out = [
        ("round", [A(1), A(511), A(512), A(513), A(1000), A(0)], P),
        ("2mb_for_1mb", [A(1000000)], P),
        ("20mb_for_10mb", [A(10000000)], P),
        ("min_large_edge", [A(10 * MiB), A(10 * MiB - 512)], P),
        ("pool_edge", [A(MiB), A(MiB + 1), A(0), F(2)], P),
        ("w4", [A(512 * KiB)] * 4 + [F(1), F(2), A(MiB)], P),
        ("w5", [A(768 * KiB), A(256 * KiB), A(512 * KiB), A(512 * KiB), F(0), F(2), A(512 * KiB), A(768 * KiB)], P),
        ("w6", [A(256 * KiB)] * 8 + [F(0), F(4), A(256 * KiB), F(5), A(512 * KiB)], P),
        ("w7", [A(11 * MiB), F(0), A(3 * MiB)], P),
        ("w8", [A(MiB), F(0), A(19 * MiB)], cap(20 * MiB)),
        ("w8oom", [A(MiB), F(0), A(19 * MiB)], cap(20 * MiB - 1)),
        ("w8b", [A(MiB), A(19 * MiB)], cap(21 * MiB)),
        ("w9", [A(MiB)] * 5, P),
        ("w10", [A(12 * MiB), F(0), A(10 * MiB), F(2), A(14 * MiB), F(4), A(12 * MiB), F(6), A(16 * MiB), F(8)], P),
        ("w11", [A(MiB), F(0), A(512), F(2), A(700 * KiB), F(4), A(MiB), F(6), A(1), F(8)], P),
        ("w13", [A(3 * MiB), A(2 * MiB), A(2 * MiB), F(0), A(2 * MiB), F(1), A(3 * MiB), A(13 * MiB)], P),
        ("w13pt", [A(3 * MiB), A(2 * MiB), A(2 * MiB), F(0), A(2 * MiB), F(1), A(3 * MiB), A(13 * MiB)], PT),
        ("w14a", [A(MiB), A(MiB - 512), A(512)], P),
        ("w14b", [A(19 * MiB)], PT),
        ("w14c", [A(19 * MiB), F(0), A(20 * MiB)], PT),
        ("bad_h_ge_e", [F(0)], P),
        ("bad_self", [A(512), F(1)], P),
        ("bad_double", [A(512), F(0), F(0)], P),
        ("bad_double_noop", [A(0), F(0), F(0)], P),
        ("bad_free_of_free", [A(512), A(1024), F(1), F(2)], P),
        ("bad_bits", [A(512), F(0) | (1 << 40)], P),
        ("bad_size", [A((1 << 48) + 1)], P),
        ("bad_forward", [A(512), A(512), F(1), F(5)], P),
        ("max_request", [A(1 << 48)], P),
        ("stop_keeps_state", [A(3 * MiB), A(MiB), F(1), F(7)], P),
        ("empty", [], P),
    ]
    return out
