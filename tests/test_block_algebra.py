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


# ---------------------------------------------------------------- reset path kept
# With the reset's dependence on the membrane kept in the gradient, the
# membrane eligibility V becomes a per-synapse state with the binary
# presynaptic value p_s as its input.  Per step s (v = V + p_s):
#     e = psi_s (v - beta A);  E = kappa E + e;  g += L_s E;
#     A' = e + rho A;  V' = alpha v - thr e,
# the same as (alpha - thr psi) v + thr beta psi A and psi v + (rho - beta psi) A.
# Over a block each output Y in {V, A, E, g} is linear in the block-start
# state and in the p_s.  The backward (adjoint) pass gives, per output, the
# sensitivity (lV, lA, lE) to the state before step s; p_s enters where V
# does, so its coefficient is lV at step s.
def step_by_step_rt(V0, A0, E0, p, psi, L, kappa, rho, beta, alpha, thr):
    V, A, E, g = V0, A0, E0, 0.0
    for s in range(len(psi)):
        v = V + p[s]
        e = psi[s] * (v - beta * A)
        E = kappa * E + e
        g += L[s] * E
        V, A = (alpha - thr * psi[s]) * v + thr * beta * psi[s] * A, psi[s] * v + (rho - beta * psi[s]) * A
    return V, A, E, g


def block_coefficients_rt(psi, L, kappa, rho, beta, alpha, thr):
    """Per output Y: C_Y[s] (coefficient of p_s) and (lV, lA, lE) at s = 0."""
    K = len(psi)
    out = {}
    for Y, term in (("V", (1.0, 0.0, 0.0)), ("A", (0.0, 1.0, 0.0)), ("E", (0.0, 0.0, 1.0)),
                    ("g", (0.0, 0.0, 0.0))):
        aV, aA, aE = term
        C = np.zeros(K)
        for s in range(K - 1, -1, -1):
            tE = aE + (L[s] if Y == "g" else 0.0)
            w = psi[s] * (aA + tE - thr * aV)
            aV, aA, aE = alpha * aV + w, rho * aA - beta * w, kappa * tE
            C[s] = aV
        out[Y] = (C, (aV, aA, aE))
    return out


def block_form_rt(V0, A0, E0, p, psi, L, kappa, rho, beta, alpha, thr):
    co = block_coefficients_rt(psi, L, kappa, rho, beta, alpha, thr)
    res = []
    for Y in ("V", "A", "E", "g"):
        C, (lV, lA, lE) = co[Y]
        res.append(p @ C + lV * V0 + lA * A0 + lE * E0)
    return tuple(res)


@pytest.mark.parametrize("beta", [0.0, 1.8])
@pytest.mark.parametrize("K", [1, 2, 5, 16, 64, 256])
def test_block_form_rt_equals_recursion(K, beta):
    rng = np.random.default_rng(2000 * K + int(10 * beta))
    kappa, rho, alpha, thr = np.exp(-1 / 20), np.exp(-1 / 200), np.exp(-1 / 20), 0.6
    for _ in range(20):
        p = (rng.random(K) < 0.3).astype(float)
        psi = rng.uniform(0, 0.5, K) * (rng.random(K) < 0.6)
        L = rng.normal(0, 1, K)
        V0, A0, E0 = rng.normal(0, 3, 3)
        ref = step_by_step_rt(V0, A0, E0, p, psi, L, kappa, rho, beta, alpha, thr)
        got = block_form_rt(V0, A0, E0, p, psi, L, kappa, rho, beta, alpha, thr)
        for r, x in zip(ref, got):
            assert abs(r - x) <= 1e-11 * (1 + abs(r)), (K, beta, ref, got)


def test_block_form_rt_structure():
    # the coefficient of V0 is that of p_0; E0 reaches E only through kappa^K
    # and never reaches V or A; with beta = 0 the adaptation eligibility
    # reaches nothing else; thr = 0 gives the reset-stopped recursion
    rng = np.random.default_rng(11)
    K, kappa, rho, alpha = 40, np.exp(-1 / 20), np.exp(-1 / 200), np.exp(-1 / 20)
    psi, L = rng.uniform(0, 0.5, K), rng.normal(0, 1, K)
    co = block_coefficients_rt(psi, L, kappa, rho, 1.8, alpha, 0.6)
    for Y in "VAEg":
        C, (lV, lA, lE) = co[Y]
        assert lV == C[0]
    assert co["V"][1][2] == 0.0 and co["A"][1][2] == 0.0
    assert co["E"][1][2] == pytest.approx(kappa ** K, rel=1e-13)
    lif = block_coefficients_rt(psi, L, kappa, rho, 0.0, alpha, 0.6)
    for Y in "VEg":
        assert lif[Y][1][1] == 0.0
    # thr = 0: E and g coefficients of p_s are those of zbar-based ones with
    # zbar_s = sum_{r<=s} alpha^(s-r) p_r (the reset-stopped recursion above)
    p = (rng.random(K) < 0.3).astype(float)
    zbar = np.array([sum(alpha ** (s - r) * p[r] for r in range(s + 1)) for s in range(K)])
    ref = step_by_step(0.0, 0.0, zbar, psi, L, kappa, rho, 1.8)
    V, A, E, g = block_form_rt(0.0, 0.0, 0.0, p, psi, L, kappa, rho, 1.8, alpha, 0.0)
    assert E == pytest.approx(ref[0], rel=1e-12) and A == pytest.approx(ref[1], rel=1e-12)
    assert g == pytest.approx(ref[2], rel=1e-12)


# ---------------------------------------------------------------- binary-input form
# zbar_s = alpha^(s+1) Z + sum_{r<=s} alpha^(s-r) p_r, with Z the filter at the
# block's start, so every contraction with zbar is one with the binary p
# against the alpha-filtered coefficients X'_r = sum_{s>=r} alpha^(s-r) X_s
# (a backward recursion X'_r = X_r + alpha X'_{r+1}) plus Z alpha X'_0.
def primed(X, alpha):
    out = np.zeros_like(X)
    acc = 0.0
    for r in range(len(X) - 1, -1, -1):
        acc = X[r] + alpha * acc
        out[r] = acc
    return out


@pytest.mark.parametrize("beta", [0.0, 1.8])
@pytest.mark.parametrize("K", [1, 3, 16, 100, 256])
def test_binary_input_form_equals_recursion(K, beta):
    rng = np.random.default_rng(3000 * K + int(10 * beta))
    kappa, rho, alpha = np.exp(-1 / 20), np.exp(-1 / 200), np.exp(-1 / 20)
    for _ in range(10):
        p = (rng.random(K) < 0.3).astype(float)
        Z = rng.uniform(0, 5)
        zbar = np.zeros(K)
        z = Z
        for s in range(K):
            z = alpha * z + p[s]
            zbar[s] = z
        psi = rng.uniform(0, 0.3, K) * (rng.random(K) < 0.6)
        L = rng.normal(0, 1, K)
        E0, A0 = rng.normal(0, 3, 2)
        ref = step_by_step(E0, A0, zbar, psi, L, kappa, rho, beta)
        U, V, H, c, q, P, D = block_coefficients(psi, L, kappa, rho, beta)
        Up, Vp, Hp = primed(U, alpha), primed(V, alpha), primed(H, alpha)
        got = (kappa ** K * E0 + P * A0 + p @ Up + Z * alpha * Up[0],
               D * A0 + p @ Vp + Z * alpha * Vp[0],
               c * E0 + q * A0 + p @ Hp + Z * alpha * Hp[0])
        for r, x in zip(ref, got):
            assert abs(r - x) <= 1e-11 * (1 + abs(r)), (K, beta, ref, got)


# ---------------------------------------------------------------- any linear two-component neuron
# A neuron step linear in its state, h = A h_prev + b I + r z_prev with the
# spike argument c . h - thr, has the per-synapse recursion (sigma: the
# stored eligibility before the next input, H_I = A + psi_prev r c^T, F = b p)
#     eps = sigma + b p_s;  e = psi_s (c . eps);  E = kappa E + e;  g += L_s E;
#     sigma' = A eps + r e.
# The adjoint pass of the eligibility kernel's coefficients is generic in
# (A, b, r, c); with A = diag(alpha, rho), b = (1, 0), r = (-thr, 1),
# c = (1, -beta) it is the reset-kept recursion above, and the two-compartment
# neuron has A = [[alpha, g], [0, alpha_d]], b = (0, 1), r = (0 or -thr, q),
# c = (1, 0).
def step_by_step_gen(S0, E0, p, psi, L, kappa, A, b, r, c):
    S, E, g = np.array(S0, float), E0, 0.0
    for s in range(len(psi)):
        eps = S + b * p[s]
        e = psi[s] * (c @ eps)
        E = kappa * E + e
        g += L[s] * E
        S = A @ eps + r * e
    return S[0], S[1], E, g


def block_form_gen(S0, E0, p, psi, L, kappa, A, b, r, c):
    K = len(psi)
    res = []
    for Y in ("S0", "S1", "E", "g"):
        l = np.array([1.0 if Y == "S0" else 0.0, 1.0 if Y == "S1" else 0.0])
        lE = 1.0 if Y == "E" else 0.0
        C = np.zeros(K)
        for s in range(K - 1, -1, -1):
            tE = lE + (L[s] if Y == "g" else 0.0)
            le = tE + r @ l
            w = psi[s] * le
            l = A.T @ l + c * w
            lE = kappa * tE
            C[s] = b @ l
        res.append(p @ C + l @ np.asarray(S0) + lE * E0)
    return tuple(res)


@pytest.mark.parametrize("K", [1, 3, 16, 100, 256])
def test_generic_block_form_equals_recursion(K):
    rng = np.random.default_rng(77 + K)
    kappa = np.exp(-1 / 20)
    for _ in range(10):
        A = rng.normal(0, 0.5, (2, 2)) + np.diag([0.5, 0.5])
        b, r, c = rng.normal(0, 1, 2), rng.normal(0, 1, 2), rng.normal(0, 1, 2)
        p = (rng.random(K) < 0.3).astype(float)
        psi = rng.uniform(0, 0.5, K) * (rng.random(K) < 0.6)
        L = rng.normal(0, 1, K)
        S0, E0 = rng.normal(0, 3, 2), rng.normal(0, 3)
        ref = step_by_step_gen(S0, E0, p, psi, L, kappa, A, b, r, c)
        got = block_form_gen(S0, E0, p, psi, L, kappa, A, b, r, c)
        scale = 1 + max(abs(x) for x in ref)
        for x, y in zip(ref, got):
            assert abs(x - y) <= 1e-10 * scale, (K, ref, got)


def test_generic_form_reduces_to_the_reset_kept_recursion():
    rng = np.random.default_rng(5)
    K, kappa, rho, alpha, thr, beta = 40, np.exp(-1 / 20), np.exp(-1 / 200), np.exp(-1 / 20), 0.6, 1.8
    A, b = np.diag([alpha, rho]), np.array([1.0, 0.0])
    r, c = np.array([-thr, 1.0]), np.array([1.0, -beta])
    p = (rng.random(K) < 0.3).astype(float)
    psi = rng.uniform(0, 0.5, K)
    L = rng.normal(0, 1, K)
    V0, A0, E0 = rng.normal(0, 3, 3)
    ref = step_by_step_rt(V0, A0, E0, p, psi, L, kappa, rho, beta, alpha, thr)
    got = step_by_step_gen([V0, A0], E0, p, psi, L, kappa, A, b, r, c)
    for x, y in zip(ref, got):
        assert abs(x - y) <= 1e-12 * (1 + abs(x))
