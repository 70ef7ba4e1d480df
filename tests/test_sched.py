"""Deficit token-budget admission (Sec. 4.1, Alg. 1): the library's native
rule against the paper's worked example, the guarantees the paper states for
it, and a closed-form restatement of the rule (oracle/deficit.py: the longest
head of the queue whose prefix sum fits the budget)."""
import ctypes
import os

import numpy as np
import pytest

from oracle import deficit as ref
from paper_2607_04206_amd._lib import SangamError, check, lib

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "deficit_three_iterations.txt")


def admit(tau, decodes, waiting, deficit):
    """The library's sangam_deficit_admit: (admitted, new deficit)."""
    w = np.asarray(waiting, np.int64)
    d = ctypes.c_int64(deficit)
    n = ctypes.c_int32(-1)
    check(lib.sangam_deficit_admit(int(tau), int(sum(decodes)), len(decodes),
                                   w.ctypes.data if len(w) else None, len(w), ctypes.byref(d),
                                   ctypes.byref(n)))
    return n.value, d.value


def load_golden():
    tau, steps = None, []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        f = line.split()
        if f[0] == "tau":
            tau = int(f[1])
        else:
            kv = dict(zip(f[0::2], f[1::2]))
            steps.append((int(kv["decodes"]), [int(x) for x in kv["waiting"].split(",")],
                          int(kv["admitted"]), int(kv["deficit"])))
    return tau, steps


@pytest.mark.parametrize("impl", ["library", "oracle"])
def test_paper_worked_example(impl):
    tau, steps = load_golden()
    deficit = 0
    for dec, waiting, want_n, want_def in steps:
        f = admit if impl == "library" else ref.admit
        n, deficit = f(tau, [dec], waiting, deficit)
        assert (n, deficit) == (want_n, want_def)


def simulate(f, tau, decode_seq, arrivals, rng_seed=0):
    """Drive an admission function over a stream: decode_seq[t] lists the
    decodes of iteration t, arrivals[t] the prefills arriving before it."""
    queue, deficit, log = [], 0, []
    for t, dec in enumerate(decode_seq):
        queue.extend(arrivals[t])
        before = list(queue)
        n, deficit = f(tau, dec, queue, deficit)
        log.append((dec, before, n, deficit))
        del queue[:n]
    return log


def random_stream(seed, T=400, tau=1024, max_decodes=40, min_decodes=0):
    rng = np.random.default_rng(seed)
    decode_seq = [[32] * int(rng.integers(min_decodes, max_decodes + 1)) for _ in range(T)]
    arrivals = [[int(x) for x in rng.integers(100, 3 * tau, size=rng.poisson(0.4))] for _ in range(T)]
    return tau, decode_seq, arrivals


@pytest.mark.parametrize("seed", range(6))
def test_library_matches_closed_form(seed):
    tau, decs, arr = random_stream(seed)
    assert simulate(admit, tau, decs, arr) == simulate(ref.admit, tau, decs, arr)


@pytest.mark.parametrize("seed", range(4))
def test_library_matches_closed_form_single_iterations(seed):
    # single iterations over a wide range: budgets below zero (decodes over
    # tau), idle microbatches, oversized heads, carries larger than tau
    rng = np.random.default_rng(100 + seed)
    for _ in range(2000):
        tau = int(rng.integers(0, 4096))
        dec = [32] * int(rng.integers(0, 80))
        waiting = [int(x) for x in rng.integers(1, 5000, size=int(rng.integers(0, 6)))]
        deficit = int(rng.integers(0, 6000))
        assert admit(tau, dec, waiting, deficit) == ref.admit(tau, dec, waiting, deficit), \
            (tau, len(dec), waiting, deficit)


@pytest.mark.parametrize("seed", range(6))
def test_per_iteration_rules(seed):
    tau, decs, arr = random_stream(seed)
    for dec, before, n, deficit in simulate(admit, tau, decs, arr):
        # admission takes a prefix of the queue in arrival order (never skips)
        assert 0 <= n <= len(before)
        if not before:
            assert n == 0 and deficit == 0  # decode-only iteration clears the carry
            continue
        if len(dec) == 0:
            assert n >= 1  # the idle rule: an empty microbatch admits the head prefill


@pytest.mark.parametrize("seed", range(6))
def test_amortized_bound(seed):
    # the paper's bound: over a busy period of W iterations with prefills
    # waiting throughout, admitted prefill tokens <= W tau - sum D_t. It holds
    # exactly while the decodes of an iteration fit tau and the microbatch is
    # never empty (the idle rule, there for liveness, may exceed it by the one
    # oversized prefill it admits; decodes beyond tau leave a negative budget
    # that the carry does not repay)
    tau, decs, arr = random_stream(seed, max_decodes=32, min_decodes=1)
    W = admitted = decoded = 0
    for dec, before, n, deficit in simulate(admit, tau, decs, arr):
        if not before:
            W = admitted = decoded = 0
            continue
        W += 1
        admitted += sum(before[:n])
        decoded += sum(dec)
        assert admitted <= W * tau - decoded
        assert admitted + deficit == W * tau - decoded  # the carry is exactly the unspent budget


def test_decodes_never_displaced_and_budget_respected():
    # decodes above tau leave no budget: no prefill joins a non-empty microbatch
    assert admit(1024, [32] * 40, [1], 0) == (0, 0)
    # with the carry a prefill that does not fit tau alone is admitted
    assert admit(1024, [32] * 10, [1000], 400) == (1, 1024 - 320 + 400 - 1000)
    # an oversized prefill enters an idle system (liveness) and leaves no carry
    assert admit(1024, [], [5000, 10], 0) == (1, 0)
    # but not a busy one
    assert admit(1024, [32], [5000], 0) == (0, 992)


def test_rejects_bad_arguments():
    d, n = ctypes.c_int64(0), ctypes.c_int32(0)
    w = np.asarray([5, 0], np.int64)
    st = lib.sangam_deficit_admit(1024, 0, 0, w.ctypes.data, 2, ctypes.byref(d), ctypes.byref(n))
    assert st == -1
    st = lib.sangam_deficit_admit(-1, 0, 0, None, 0, ctypes.byref(d), ctypes.byref(n))
    assert st == -1
    st = lib.sangam_deficit_admit(1024, 0, 0, None, 0, None, ctypes.byref(n))
    assert st == -1
    d.value = -5
    st = lib.sangam_deficit_admit(1024, 0, 0, None, 0, ctypes.byref(d), ctypes.byref(n))
    assert st == -1
