"""Precision of the contraction operands of the eligibility kernel (CPU).

The block coefficients that multiply the binary presynaptic values are
carried as scaled fp16 pairs: a row of values x_s (one batch element and
neuron, the steps of a block) is multiplied by a power of two 2^e that puts
its largest magnitude in [2^13, 2^14), and each scaled value becomes
hi = fp16(x 2^e) and lo = fp16(x 2^e - hi).  The matrix cores then sum
hi p + lo p in fp32 (p is 0 or 1, exact in fp16).  This file restates that
encoding in numpy and checks its error on adversarial rows: a pseudo-
derivative that is zero for most steps and a learning signal that spans many
decades within the block, so that most entries are tiny next to the row's
largest one.

The bound: |x 2^e - hi| <= ulp(hi)/2 <= 4, so lo has an exponent <= 2 and
|x 2^e - hi - lo| <= 2^-9, i.e. the pair keeps every entry to within
2^-22 of the row's largest magnitude (absolute, not relative), and a sum
over the row of p_s x_s to within 2^-22 max|x| times the number of terms.
"""
import numpy as np
import pytest


def pair_encode(x):
    """Row-wise scaled fp16 pairs of a float32 array [rows, steps]."""
    x = np.asarray(x, dtype=np.float32)
    m = np.abs(x).max(axis=1)
    _, k = np.frexp(m)                      # m in [2^(k-1), 2^k)
    e = np.where(m > 0, np.clip(14 - k, -100, 100), 0)
    scale = np.ldexp(np.float32(1), e).astype(np.float32)[:, None]
    xs = (x * scale).astype(np.float32)
    hi = xs.astype(np.float16)
    lo = (xs - hi.astype(np.float32)).astype(np.float16)
    return hi, lo, scale


def pair_decode(hi, lo, scale):
    return (hi.astype(np.float64) + lo.astype(np.float64)) / scale.astype(np.float64)


def adversarial_rows(rng, rows=512, steps=256, decades=10.0, active=0.15):
    """Coefficient-like rows psi_s * M_s with psi zero on most steps and M
    spanning `decades` decades over the block, then alpha-filtered backwards
    (X'_r = X_r + alpha X'_{r+1}) like the operands of the kernel."""
    psi = np.where(rng.random((rows, steps)) < active, rng.uniform(0.0, 0.3, (rows, steps)), 0.0)
    logm = np.linspace(0.0, -decades, steps)[None, :] + rng.normal(0, 0.5, (rows, steps))
    M = rng.choice([-1.0, 1.0], (rows, steps)) * 10.0 ** logm
    X = psi * M
    alpha = np.float64(np.float32(np.exp(-1 / 20)))
    Xf = np.zeros_like(X)
    acc = np.zeros(rows)
    for s in range(steps - 1, -1, -1):
        acc = X[:, s] + alpha * acc
        Xf[:, s] = acc
    return Xf.astype(np.float32)


@pytest.mark.parametrize("decades", [2.0, 8.0, 12.0])
def test_pair_error_is_bounded_by_the_row_maximum(decades):
    rng = np.random.default_rng(int(decades))
    x = adversarial_rows(rng, decades=decades)
    hi, lo, scale = pair_encode(x)
    rmax = np.abs(x.astype(np.float64)).max(axis=1, keepdims=True)
    err = np.abs(pair_decode(hi, lo, scale) - x.astype(np.float64))
    assert np.all(err <= 2.0 ** -22 * rmax)
    # the pair is far better than one fp16 word: dropping lo costs ~2^-11
    err1 = np.abs(hi.astype(np.float64) / scale - x.astype(np.float64))
    assert err1.max() > 2.0 ** 6 * err.max()
    # entries many decades below the row maximum keep only absolute precision
    small = np.abs(x) < 1e-6 * rmax
    assert small.any()


@pytest.mark.parametrize("decades", [8.0, 12.0])
def test_pair_contraction_meets_the_gradient_bar(decades):
    # sum_s p_s x_s for binary p over the block, as the matrix cores form it
    # (hi p + lo p with fp32 accumulation, 32 terms per instruction), against
    # the exact sum; the relative L2 error over all (row, input) pairs stays
    # far below the 1e-4 parity bar, and each entry within the absolute bound.
    rng = np.random.default_rng(100 + int(decades))
    x = adversarial_rows(rng, rows=256, decades=decades)
    p = (rng.random((64, x.shape[1])) < 0.03).astype(np.float32)    # ~3% presynaptic activity
    hi, lo, scale = pair_encode(x)
    exact = p.astype(np.float64) @ x.astype(np.float64).T
    acc = np.zeros((64, x.shape[0]), dtype=np.float32)
    for c in range(0, x.shape[1], 16):                    # one 16-step chunk per instruction
        part = (p[:, c:c + 16] @ hi[:, c:c + 16].astype(np.float32).T).astype(np.float32)
        part = (part + p[:, c:c + 16] @ lo[:, c:c + 16].astype(np.float32).T).astype(np.float32)
        acc = (acc + part).astype(np.float32)
    got = acc.astype(np.float64) / scale[:, 0][None, :].astype(np.float64)
    rmax = np.abs(x.astype(np.float64)).max(axis=1)
    nterms = p.sum(axis=1, keepdims=True)
    assert np.all(np.abs(got - exact) <= (2.0 ** -22 + 2.0 ** -23 * 16) * rmax[None, :] * (nterms + 1))
    rel = np.linalg.norm(got - exact) / np.linalg.norm(exact)
    assert rel < 1e-6, rel
