"""Pins of oracle.stabilize (Appendix C) against numpy's SVD and inverse.

The appendix states what fix-singular-value must achieve: the chosen singular
value of U becomes sigma_star, the singular vectors and the other singular
values do not change, W = V U is unchanged (so is Q = W^T W) and U^{-T} stays
the inverse transpose of U.  Each test checks one of these facts with an
independent routine (SVD, inverse), on matrices built with a known spectrum.
The last test plants plausible mistakes and checks that the pins catch them.
"""
import numpy as np
import pytest

from oracle import factored, stabilize


def _orth(rng, d):
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))


def _state(sigmas, D=30, seed=3):
    rng = np.random.default_rng(seed)
    d = len(sigmas)
    U = _orth(rng, d) @ np.diag(sigmas) @ _orth(rng, d).T
    V = rng.uniform(-0.5, 0.5, size=(D, d))
    return factored.FactoredState.from_initial(V, U)


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def _check_fix(st0, st1, k_moved, s_before, target):
    """The appendix's claims about one correction, checked with SVD and inverse."""
    Ub0, s0, Vb0 = np.linalg.svd(st0.U)
    Ub1, s1, Vb1 = np.linalg.svd(st1.U)
    want = np.array(s_before, dtype=float)
    want[k_moved] = target
    np.testing.assert_allclose(np.sort(s1), np.sort(want), rtol=1e-12, atol=1e-14)
    # same singular subspaces: |U_b1^T U_b0| is a permutation matrix
    P = np.abs(Ub1.T @ Ub0)
    np.testing.assert_allclose(np.sort(P.max(axis=1)), np.ones(len(s1)), atol=1e-9)
    assert _rel(st1.V @ st1.U, st0.V @ st0.U) < 1e-13        # W unchanged
    np.testing.assert_allclose(st1.UinvT, np.linalg.inv(st1.U).T, rtol=0, atol=1e-10)
    W1 = st1.V @ st1.U
    assert _rel(W1.T @ W1, st0.Q) < 1e-12                     # Q still W^T W


def _copy(st):
    return factored.FactoredState(V=st.V.copy(), U=st.U.copy(), UinvT=st.UinvT.copy(),
                                  Q=st.Q.copy(), c=st.c.copy(), s=st.s.copy())


@pytest.mark.parametrize("k", [0, 3, 6])
def test_fix_singular_value_moves_only_that_value(k):
    sig = [7.0, 3.0, 2.0, 1.5, 0.5, 0.1, 1e-3]
    st0 = _state(sig)
    st1 = _copy(st0)
    Ub, s, _ = np.linalg.svd(st1.U)
    alpha, beta = stabilize.fix_singular_value(st1, float(s[k]), Ub[:, k], 1.0)
    _check_fix(st0, st1, k, s, 1.0)
    # with sigma_star = 1: 1 + alpha = 1 / sigma and beta = sigma - 1
    assert abs((1.0 + alpha) - 1.0 / s[k]) < 1e-12 * (1.0 / s[k])
    assert abs(beta - (s[k] - 1.0)) < 1e-12


def test_fix_to_another_target():
    st0 = _state([4.0, 2.0, 1.0, 0.25])
    st1 = _copy(st0)
    Ub, s, _ = np.linalg.svd(st1.U)
    stabilize.fix_singular_value(st1, float(s[1]), Ub[:, 1], 0.5)
    _check_fix(st0, st1, 1, s, 0.5)


def test_power_iteration_matches_svd():
    rng = np.random.default_rng(11)
    d = 9
    A = _orth(rng, d) @ np.diag([5.0, 2.5, 1.2, 1, 1, 0.9, 0.5, 0.3, 0.2]) @ _orth(rng, d).T
    sigma, u = stabilize.top_left_singular_pair(A, 128, np.ones(d))
    Ub, s, _ = np.linalg.svd(A)
    assert abs(sigma - s[0]) < 1e-12 * s[0]
    assert abs(abs(u @ Ub[:, 0]) - 1.0) < 1e-12


def test_power_iteration_equals_repeated_squaring():
    """2^k power iterations equal k squarings of A A^T applied to x0 (exact
    arithmetic; fp64 here): the GPU library takes the squaring route."""
    rng = np.random.default_rng(5)
    d = 12
    A = _orth(rng, d) @ np.diag(np.linspace(3.0, 0.5, d)) @ _orth(rng, d).T
    x0 = np.ones(d)
    _, u_it = stabilize.top_left_singular_pair(A, 2 ** 6, x0)
    G = A @ A.T
    for _ in range(6):
        G = G / np.trace(G)
        G = G @ G
    x = G @ x0
    u_sq = x / np.linalg.norm(x)
    np.testing.assert_allclose(u_sq, u_it, rtol=0, atol=1e-12)


def test_stabilize_power_restores_range_and_keeps_W():
    sig = [300.0, 1.0, 1.0, 1.0, 0.8, 5e-4, 1e-4]
    st0 = _state(sig)
    st1 = _copy(st0)
    rounds = stabilize.stabilize_power(st1, 1e-3, 100.0, 128, 4, np.ones(len(sig)))
    s1 = np.linalg.svd(st1.U, compute_uv=False)
    assert s1.min() >= 1e-3 and s1.max() <= 100.0
    assert [r[2] for r in rounds] == [True, True, False, True, False]
    assert _rel(st1.V @ st1.U, st0.V @ st0.U) < 1e-12
    np.testing.assert_allclose(st1.UinvT, np.linalg.inv(st1.U).T, rtol=0, atol=1e-9)
    # the corrected values went to 1; the others did not move
    np.testing.assert_allclose(np.sort(s1), np.sort([1.0, 1, 1, 1, 0.8, 1, 1]), rtol=1e-9)


def test_stabilize_svd_and_power_agree():
    sig = [250.0, 1.0, 0.7, 2e-4]
    st_a, st_b = _state(sig), _state(sig)
    fixed = stabilize.stabilize_svd(st_a, 1e-3, 100.0)
    assert fixed == [0, 3]
    stabilize.stabilize_power(st_b, 1e-3, 100.0, 128, 3, np.ones(4))
    assert _rel(st_b.U, st_a.U) < 1e-9
    assert _rel(st_b.V, st_a.V) < 1e-9


def test_in_range_changes_nothing():
    st0 = _state([2.0, 1.0, 0.5])
    st1 = _copy(st0)
    rounds = stabilize.stabilize_power(st1, 1e-3, 100.0, 64, 2, np.ones(3), reinvert_mode=0)
    assert [r[2] for r in rounds] == [False, False]
    np.testing.assert_array_equal(st1.U, st0.U)
    np.testing.assert_array_equal(st1.V, st0.V)
    np.testing.assert_array_equal(st1.UinvT, st0.UinvT)


def test_planted_mistakes_are_caught():
    """Plausible slips in fix-singular-value each break one of the pins."""
    st0 = _state([6.0, 1.0, 0.2, 1e-3])
    Ub, s, Vb = np.linalg.svd(st0.U)
    k = 3

    def wrong_beta_sign(st, sigma, u):
        a = (1.0 - sigma) / sigma
        b = +a / (1.0 + a)
        Uinv = st.UinvT.T
        wu, wi = st.U.T @ u, Uinv @ u
        st.U = st.U + a * np.outer(u, wu)
        st.V = st.V + b * np.outer(st.V @ u, u)
        st.UinvT = st.UinvT + b * np.outer(u, wi)

    def new_inverse_used(st, sigma, u):
        a = (1.0 - sigma) / sigma
        b = -a / (1.0 + a)
        st.U = st.U + a * np.outer(u, st.U.T @ u)
        st.V = st.V + b * np.outer(st.V @ u, u)
        st.UinvT = st.UinvT + b * np.outer(u, np.linalg.inv(st.U) @ u)

    def right_vector(st, sigma, u_left):
        stabilize.fix_singular_value(st, sigma, Vb[k], 1.0)

    for bad in (wrong_beta_sign, new_inverse_used, right_vector):
        st1 = _copy(st0)
        bad(st1, float(s[k]), Ub[:, k])
        with pytest.raises(AssertionError):
            _check_fix(st0, st1, k, s, 1.0)
