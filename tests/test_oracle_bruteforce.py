"""Brute force on tiny inputs: the C++ oracle against the Python interval-list
model on every trace of <= 2 blocks over the boundary alphabet, on every
3-block trace over a reduced alphabet, and on a seeded sample of the full
3-block set, under the paper parameters, the PYTORCH_LIKE split preset and
small device capacities that force reclaim and OOM."""
import numpy as np
import pytest

import oracle
from bf_model import run as bf_run
from bf_traces import enumerate_traces, to_csr
from evw import KiB, MiB

PARAMS = {
    "paper": oracle.paper_params(),
    "pytorch_like": oracle.pytorch_like_params(),
    "cap22": oracle.paper_params(device_capacity_bytes=22 * MiB),
    "cap20": oracle.paper_params(device_capacity_bytes=20 * MiB),
    "cap14": oracle.paper_params(device_capacity_bytes=14 * MiB),
    "cap40": oracle.paper_params(device_capacity_bytes=40 * MiB),
    "cap4": oracle.paper_params(device_capacity_bytes=4 * MiB),
}
REDUCED = [0, 513, 256 * KiB, MiB, MiB + 1, 13 * MiB]


def check_batch(traces, params):
    ev, off = to_csr(traces)
    rc, out, ser = oracle.replay(ev, off, params, series=True)
    assert rc == 0
    for t, tr in enumerate(traces):
        bres, bser = bf_run(tr, params)
        got = {k: int(out[t][k]) for k in bres}
        assert got == bres, (tr, got, bres)
        assert [int(x) for x in ser[off[t]:off[t + 1]]] == bser, tr


@pytest.mark.parametrize("pname", list(PARAMS))
def test_upto_two_blocks_exhaustive(pname):
    check_batch(enumerate_traces(2), PARAMS[pname])


@pytest.mark.parametrize("pname", ["paper", "pytorch_like", "cap22", "cap20", "cap14"])
def test_three_blocks_reduced_alphabet(pname):
    check_batch(enumerate_traces(3, alphabet=REDUCED), PARAMS[pname])


def test_three_blocks_sample():
    check_batch(enumerate_traces(3, sample=4000, seed=1), PARAMS["paper"])
    check_batch(enumerate_traces(3, sample=1500, seed=2), PARAMS["cap40"])


def test_statuses_are_exercised():
    """The enumeration really reaches OOM and reclaim under the small capacities."""
    traces = enumerate_traces(3, alphabet=REDUCED)
    ev, off = to_csr(traces)
    for pname in ("cap20", "cap14"):
        _, out, _ = oracle.replay(ev, off, PARAMS[pname])
        assert (out["status"] == 1).sum() > 100, pname
        assert ((out["segments_released"] > 0) & (out["status"] == 0)).sum() > 100, pname
        assert (out["status"] == 0).sum() > 1000, pname
