"""Appendix C numerical stabilisation, plainly, in fp64 (test infrastructure only).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The factored state (V, U, U^{-T}, Q) of `oracle.factored` represents W = V U.
Appendix C keeps U well conditioned without the O(D d^2) pristine restore:
it corrects only the singular values of U that leave a safe range
[sigma_low, sigma_high], each with a rank-one change of U, U^{-T} and V that
leaves W = V U (hence Q = W^T W) unchanged.

Functions
  fix_singular_value       moves one singular value sigma of U, with left singular
                           vector u, to sigma_star (a symmetric rank-one left
                           factor on U, its inverse on V).
  stabilize_svd            the appendix's procedure with a full SVD of U: every
                           singular value outside the range is moved to 1.
  top_left_singular_pair   the power iteration the appendix proposes instead of the
                           SVD: the largest singular value of a d x d matrix A and
                           its left singular vector, by x <- A A^T x / ||A A^T x||.
  reinvert                 U^{-T} recomputed from U (the appendix does this before
                           every check).
  stabilize_power          the appendix's loop: find the smallest singular value of
                           U (power iteration on U^{-T}, whose largest singular
                           value is 1 / sigma_min(U) with the same left singular
                           vector), correct it while it is below the range, then
                           the same for the largest (power iteration on U).

Pins: every function here is checked against numpy's SVD / inverse and the
invariants the appendix states (W, Q unchanged; U^{-T} stays the inverse; only
the chosen singular value moves) in tests/test_stabilize_pins.py.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

from .factored import FactoredState


def fix_singular_value(st: FactoredState, sigma: float, u: np.ndarray, sigma_star: float = 1.0):
    """Move the singular value sigma of U (left singular vector u, unit norm) to sigma_star.

    With U = sum_k s_k u_k v_k^T, left-multiplying U by L = I + alpha u u^T,
    alpha = sigma_star / sigma - 1, scales the term of u by 1 + alpha and leaves
    every other singular value and every singular vector alone.  W = V U stays
    the same when V is right-multiplied by L^{-1} = I + beta u u^T with
    beta = -alpha / (1 + alpha) (Sherman-Morrison for a rank-one change of the
    identity), and since L is symmetric the new U^{-T} is L^{-1} U^{-T}.
    Each of the three products is applied as a rank-one correction, so V costs
    O(D d).  Applied in place; returns (alpha, beta).
    """
    u = np.asarray(u, dtype=np.float64)
    alpha = sigma_star / sigma - 1.0
    beta = -alpha / (1.0 + alpha)
    # L U = U + alpha u (u^T U);  L^{-1} U^{-T} = U^{-T} + beta u (u^T U^{-T});
    # V L^{-1} = V + beta (V u) u^T.  Row vectors u^T U and u^T U^{-T} from the old state.
    uU = u @ st.U
    uUinvT = u @ st.UinvT
    st.U = st.U + alpha * np.outer(u, uU)
    st.UinvT = st.UinvT + beta * np.outer(u, uUinvT)
    st.V = st.V + beta * np.outer(st.V @ u, u)
    return alpha, beta


def stabilize_svd(st: FactoredState, sigma_low: float, sigma_high: float) -> List[int]:
    """The appendix's procedure with a full SVD: fix every out-of-range singular value.

    One SVD serves all corrections: a correction changes only its own singular
    value, so the other singular values and vectors stay valid.  Returns the
    indices (in decreasing-sigma order) that were corrected.
    """
    Ub, s, _ = np.linalg.svd(st.U)
    fixed = []
    for k in range(len(s)):
        if s[k] < sigma_low or s[k] > sigma_high:
            fix_singular_value(st, float(s[k]), Ub[:, k], 1.0)
            fixed.append(k)
    return fixed


def top_left_singular_pair(A: np.ndarray, iterations: int, x0: np.ndarray
                           ) -> Tuple[float, np.ndarray]:
    """Power iteration for the largest singular value of A and its left singular vector.

    x <- A (A^T x), normalised, `iterations` times from x0; then u = x and the
    estimate sigma = ||A^T u|| (for an exact singular vector, A^T u = sigma v).
    """
    x = np.asarray(x0, dtype=np.float64)
    x = x / np.linalg.norm(x)
    for _ in range(iterations):
        x = A @ (A.T @ x)
        x = x / np.linalg.norm(x)
    return float(np.linalg.norm(A.T @ x)), x


def reinvert(st: FactoredState) -> None:
    """U^{-T} <- (U^{-1})^T, computed from U itself."""
    st.UinvT = np.linalg.inv(st.U).T


def stabilize_power(st: FactoredState, sigma_low: float, sigma_high: float, iterations: int,
                    max_fixes: int, x0: np.ndarray, reinvert_mode: int = 1):
    """The appendix's loop with power iterations instead of the SVD.

    With reinvert_mode 2, recompute U^{-T} first (the appendix's practice).
    Then, at most max_fixes times: estimate sigma_min(U) as 1 / sigma_max(U^{-T})
    with u the top left singular vector of U^{-T} (the left singular vector of U
    for sigma_min); stop when it is not below sigma_low, else move it to 1.  Then
    the same for sigma_max(U) against sigma_high.  With reinvert_mode >= 1,
    U^{-T} is recomputed after every correction (in exact arithmetic the
    correction's own update of U^{-T} is already exact, so this changes nothing
    here; it mirrors what a finite-precision implementation must do).
    Returns a list of (end, sigma estimate, corrected) per round, end being
    "low" or "high".
    """
    rounds = []
    if reinvert_mode >= 2:
        reinvert(st)
    for _ in range(max_fixes):
        s_inv, u = top_left_singular_pair(st.UinvT, iterations, x0)
        # sigma_min(U) from the same vector: 1 / ||U^{-1} u||
        sigma = 1.0 / float(np.linalg.norm(st.UinvT.T @ u))
        go = sigma < sigma_low
        rounds.append(("low", sigma, go))
        if not go:
            break
        fix_singular_value(st, sigma, u, 1.0)
        if reinvert_mode >= 1:
            reinvert(st)
    for _ in range(max_fixes):
        sigma, u = top_left_singular_pair(st.U, iterations, x0)
        go = sigma > sigma_high
        rounds.append(("high", sigma, go))
        if not go:
            break
        fix_singular_value(st, sigma, u, 1.0)
        if reinvert_mode >= 1:
            reinvert(st)
    return rounds
