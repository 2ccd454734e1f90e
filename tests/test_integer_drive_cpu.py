"""The integer drive's exactness argument, checked on the CPU.

When every weight is k 2^-14 with integer |k| <= 32767 and a step has n active
inputs with n max|k| <= 2^24, every partial sum of its drive is an integer of
at most 2^24 in units of 2^-14, so the fp32 sum in ascending input order (what
the fp32 drive and the oracle compute) is exact and equals the integer sum of
the k times 2^-14.  The GPU relies on this to sum int16 weights as integers in
any order at such steps (and takes the fp32 drive at the others).
"""
import numpy as np
import pytest


def fp32_sequential(w_rows):
    acc = np.float32(0.0)
    for w in w_rows:
        acc = np.float32(acc + np.float32(w))
    return acc


@pytest.mark.parametrize("n_pre", [16, 956, 1724, 4096, 8292])
def test_integer_sum_equals_fp32_sequential_sum_at_the_bound(n_pre):
    rng = np.random.default_rng(n_pre)
    lim = min(32767, (2 ** 24 - 1) // n_pre)
    for trial in range(20):
        n_act = int(rng.integers(1, n_pre + 1)) if trial else n_pre   # every input active once
        k = rng.integers(-lim, lim + 1, size=n_act)
        if trial == 1:
            k[:] = lim                                   # the largest sum the bound allows
        w = (k * 2.0 ** -14).astype(np.float32)
        assert np.array_equal(w.astype(np.float64) * 2 ** 14, k)   # the weights are exact in fp32
        order = np.arange(n_act) if trial % 2 else rng.permutation(n_act)
        s_fp32 = fp32_sequential(w[order])
        s_int = np.float32(int(k.sum()) * 2.0 ** -14)
        assert s_fp32 == s_int, (n_pre, trial)


def test_past_the_bound_the_orders_can_differ():
    # weights on the grid but far past the bound: fp32 partial sums round, so
    # the fp32 sum depends on the order (why such weights take the fp32 drive)
    rng = np.random.default_rng(1)
    k = rng.integers(-(2 ** 22), 2 ** 22, size=4000)
    w = (k * 2.0 ** -14).astype(np.float32)
    sums = {float(fp32_sequential(w[rng.permutation(len(w))])) for _ in range(10)}
    assert len(sums) > 1


@pytest.mark.parametrize("maxk", [32767, 4866, 100])
def test_bound_in_active_rows(maxk):
    # n active rows with n * maxk <= 2^24: exact in any order, at the bound too
    rng = np.random.default_rng(maxk)
    n = (2 ** 24) // maxk
    for trial in range(6):
        k = rng.integers(-maxk, maxk + 1, size=n)
        if trial == 0:
            k[:] = maxk
        w = (k * 2.0 ** -14).astype(np.float32)
        order = rng.permutation(n)
        assert fp32_sequential(w[order]) == np.float32(int(k.sum()) * 2.0 ** -14)
