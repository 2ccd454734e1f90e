"""The block form of the eligibility recursion that the GPU path evaluates.

Per synapse (i, j) and batch element the recursion of Eq. (5) with the ALIF
2x2 Jacobian (Sec. III-B/C) and the kappa-filtered trace advances, per step s,
    e     = psi_s (zbar_s - beta eps)
    ebar  = kappa ebar + e
    g    += L_s ebar
    eps   = psi_s zbar_s + (rho - beta psi_s) eps.
Over a block of K steps this is linear in the block-start (ebar, eps) and in
zbar_s, with coefficients that depend on psi, L of the postsynaptic neuron
only.  The test builds those coefficients by the backward pass the GPU
coefficient kernel uses and checks the three block results against the
step-by-step recursion in float64 on random data.
"""
import numpy as np
import pytest


def step_by_step(E0, A0, zbar, psi, L, kappa, rho, beta):
    ebar, eps, g = E0, A0, 0.0
    for s in range(len(psi)):
        e = psi[s] * (zbar[s] - beta * eps)
        ebar = kappa * ebar + e
        g += L[s] * ebar
        eps = psi[s] * zbar[s] + (rho - beta * psi[s]) * eps
    return ebar, eps, g


def block_coefficients(psi, L, kappa, rho, beta):
    """Backward pass over the block: U, V, H per step and c, q, P, D."""
    K = len(psi)
    U, V, H = np.zeros(K), np.zeros(K), np.zeros(K)
    M = Mu = nx = nxu = 0.0
    Dsuf = 1.0
    for s in range(K - 1, -1, -1):
        d = rho - beta * psi[s]
        M = kappa * M + L[s]                       # sum_{t>=s} kappa^(t-s) L_t
        Mu = 1.0 if s == K - 1 else kappa * Mu     # same with a unit vector at K-1
        H[s] = psi[s] * (M - nx)
        U[s] = psi[s] * (Mu - nxu)
        V[s] = psi[s] * Dsuf                       # psi_s prod_{u>s} d_u
        nx = beta * psi[s] * M + d * nx
        nxu = beta * psi[s] * Mu + d * nxu
        Dsuf = d * Dsuf
    return U, V, H, kappa * M, -nx, -nxu, Dsuf      # c, q, P, D


def block_form(E0, A0, zbar, psi, L, kappa, rho, beta):
    U, V, H, c, q, P, D = block_coefficients(psi, L, kappa, rho, beta)
    K = len(psi)
    ebar = kappa ** K * E0 + P * A0 + zbar @ U
    eps = D * A0 + zbar @ V
    g = c * E0 + q * A0 + zbar @ H
    return ebar, eps, g


@pytest.mark.parametrize("beta", [0.0, 1.8])
@pytest.mark.parametrize("K", [1, 2, 5, 16, 64, 128])
def test_block_form_equals_recursion(K, beta):
    rng = np.random.default_rng(1000 * K + int(10 * beta))
    kappa, rho = np.exp(-1 / 20), np.exp(-1 / 200)
    for _ in range(20):
        zbar = rng.uniform(0, 20, K) * (rng.random(K) < 0.7)
        psi = rng.uniform(0, 0.3, K) * (rng.random(K) < 0.6)
        L = rng.normal(0, 1, K)
        E0, A0 = rng.normal(0, 3), rng.normal(0, 3)
        ref = step_by_step(E0, A0, zbar, psi, L, kappa, rho, beta)
        got = block_form(E0, A0, zbar, psi, L, kappa, rho, beta)
        for r, x in zip(ref, got):
            assert abs(r - x) <= 1e-12 * (1 + abs(r)), (K, beta, ref, got)


def test_lif_coefficients_drop_the_adaptation_terms():
    # beta = 0: no eps terms reach ebar or g, and U, H are psi times the
    # kappa-weighted sums of the unit vector and of L
    rng = np.random.default_rng(7)
    K, kappa, rho = 32, np.exp(-1 / 20), np.exp(-1 / 200)
    psi, L = rng.uniform(0, 0.3, K), rng.normal(0, 1, K)
    U, V, H, c, q, P, D = block_coefficients(psi, L, kappa, rho, 0.0)
    assert q == 0.0 and P == 0.0 and D == pytest.approx(rho ** K)
    Ms = np.array([sum(kappa ** (t - s) * L[t] for t in range(s, K)) for s in range(K)])
    np.testing.assert_allclose(H, psi * Ms, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(U, psi * kappa ** (K - 1 - np.arange(K)), rtol=1e-13)
    assert c == pytest.approx(kappa * Ms[0], rel=1e-13)


def test_blocks_chain():
    # two consecutive blocks through the block form == one pass step by step
    rng = np.random.default_rng(3)
    kappa, rho, beta = np.exp(-1 / 20), np.exp(-1 / 200), 1.8
    K1, K2 = 48, 80
    zbar = rng.uniform(0, 5, K1 + K2)
    psi = rng.uniform(0, 0.3, K1 + K2)
    L = rng.normal(0, 1, K1 + K2)
    ref = step_by_step(0.0, 0.0, zbar, psi, L, kappa, rho, beta)
    e1, a1, g1 = block_form(0.0, 0.0, zbar[:K1], psi[:K1], L[:K1], kappa, rho, beta)
    e2, a2, g2 = block_form(e1, a1, zbar[K1:], psi[K1:], L[K1:], kappa, rho, beta)
    assert e2 == pytest.approx(ref[0], rel=1e-12)
    assert a2 == pytest.approx(ref[1], rel=1e-12)
    assert g1 + g2 == pytest.approx(ref[2], rel=1e-12)
