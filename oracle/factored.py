"""The paper's factored representation of W, in fp64 (test infrastructure only).

TEST INFRASTRUCTURE ONLY (see the package docstring).

W is never stored: it is V U (D x d times d x d, section 3.2), and the side
matrices Q = W^T W and U^{-T} are kept up to date (section 3.3).  For the
spherical softmax in the shifted form of section 3.6 the state also carries a
row c shared by all D rows and the column sums s = W^T 1, so that
W = V U + 1 c^T (c stays zero for the other losses).  This module
exists to check the paper's algebra against the explicit definition in
`oracle.explicit`: after every step V U must equal the explicitly updated W,
Q must equal W^T W and U (U^{-T})^T must be the identity.

How the step is organised here.  Every loss this package handles has an
output gradient of the form

    dL/dO = W H A + 1 g^T + G,   A = diag(a_1 .. a_m),  G sparse on the targets,

(squared error: a_i = 2, g = 0 and G = -2 Y, eq. gradH; spherical softmax:
see `spherical_minibatch_step`; its shifted form has g != 0, see
`shifted_spherical_minibatch_step`).  For such a loss the whole update is a
function of (H, A, g, G) and the factored state, derived once in
`_factored_update`:

  * gradient wrt H       W^T dL/dO = (Q H) A + s g^T + W^T G, with
                         W^T G = U^T (V^T G) + c (1^T G) (section 3.1, eq. gradH,
                         and the remark at the end of section 3.2 that W^T y is
                         U^T (V^T y));
  * the W update         W - lr (dL/dO) H^T is reached by
                         U <- U (I - lr H A H^T)          (eq. updateU),
                         V <- V - lr G (U_new^{-T} H)^T   (eq. updateV), and
                         c <- (I - lr H A H^T) c - lr H g,
                         since V_new U_new = V U_new - lr G H^T;
  * s = W^T 1            s - lr H (dL/dO)^T 1, with
                         (dL/dO)^T 1 = A H^T s + D g + G^T 1;
  * U^{-T}               (I - lr H A H^T)^{-1} by the Woodbury identity, which
                         for one example is the Sherman-Morrison form of
                         eq. updateU-T (section 3.5 and the minibatch appendix);
  * Q                    W_new^T W_new expanded (the proof of the Q update in the
                         appendix): Q - lr (H grad^T + grad H^T) + lr^2 H N H^T
                         with N = (dL/dO)^T (dL/dO) built from m x m pieces
                         (for g != 0 also n g^T-type pieces, n = H^T s).

Functions
  FactoredState.from_initial  the initialisation of the minibatch appendix (V = W0,
                              U = U^{-T} = I, Q = V^T V), generalised to any
                              invertible U0.
  minibatch_step              squared error, any m (a_i = 2, G = -2 Y).
  spherical_minibatch_step    spherical softmax, one class per example (the paper
                              lists this loss in section 3.6 without minibatch
                              formulas; the (a, G) form above supplies them).
  shifted_spherical_minibatch_step  the same loss in the form section 3.6 prints,
                              (o_c + eps)^2 / sum_j (o_j + eps)^2 (g = eps a).
  online_step                 one example, squared error, with the rank-one
                              (Sherman-Morrison) update of U^{-T} of eq. updateU-T.
  sherman_morrison_inverse_T  eq. updateU-T on its own.
  pristine_restore            Appendix C: V <- V U, U <- I, U^{-T} <- I.

Pin status: every step function is pinned against the explicit definition
(`oracle.explicit`) after each of many steps; the squared-error step also by the
paper's own identities.  The minibatch forms of both spherical steps have no
printed values in the paper.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .explicit import dense_targets, widen


@dataclasses.dataclass
class FactoredState:
    V: np.ndarray      # D x d
    U: np.ndarray      # d x d
    UinvT: np.ndarray  # d x d, (U^{-1})^T
    Q: np.ndarray      # d x d, W^T W
    c: np.ndarray      # d, the row shared by all rows of W (W = V U + 1 c^T)
    s: np.ndarray      # d, W^T 1

    @classmethod
    def from_initial(cls, V0, U0=None) -> "FactoredState":
        """Initial state with W0 = V0 U0 (U0 = I unless given): U^{-T} = inv(U0)^T,
        Q = W0^T W0, c = 0, s = W0^T 1.  With U0 = I this is the appendix's V = W0,
        Q = V^T V."""
        V = widen(V0)
        d = V.shape[1]
        U = np.eye(d) if U0 is None else widen(U0)
        W = V @ U
        return cls(V=V, U=U, UinvT=np.linalg.inv(U).T, Q=W.T @ W, c=np.zeros(d),
                   s=W.sum(axis=0))

    def W(self) -> np.ndarray:
        return self.V @ self.U + self.c[None, :]

    def WtG(self, G: np.ndarray) -> np.ndarray:
        """W^T G for a D x m G without forming W: U^T (V^T G) + c (1^T G)."""
        return self.U.T @ (self.V.T @ G) + np.outer(self.c, G.sum(axis=0))


def _factored_update(st: FactoredState, H: np.ndarray, a: np.ndarray, G: np.ndarray,
                     QH: np.ndarray, WtG: np.ndarray, lr: float, g=None) -> np.ndarray:
    """Apply W <- W - lr (W H A + 1 g^T + G) H^T to the factored state; return
    grad_H (d x m).

    H is d x m (columns are examples), a the diagonal of A, g the m weights of
    the all-ones direction (None: zero), G the D x m sparse part of dL/dO,
    QH = Q H and WtG = W^T G (both d x m, from the state before the update).
    The new U, U^{-T}, V and Q all follow from the same rank-m change
    I - lr H A H^T  of U's right-hand side; c and s from O(m d) products.
    """
    D = st.V.shape[0]
    m = H.shape[1]
    g = np.zeros(m) if g is None else np.asarray(g, dtype=np.float64)
    A = np.diag(a)
    n = H.T @ st.s                                       # n_i = 1^T W h_i
    grad = QH @ A + np.outer(st.s, g) + WtG              # W^T dL/dO
    # N = (dL/dO)^T (dL/dO) = A H^T Q H A + A H^T W^T G + G^T W H A + G^T G
    #     + A n g^T + g n^T A + D g g^T + g (1^T G) + (G^T 1) g^T
    HtWtG = H.T @ WtG
    Gsum = G.sum(axis=0)                                 # 1^T G
    N = (A @ (H.T @ QH) @ A + A @ HtWtG + HtWtG.T @ A + G.T @ G
         + np.outer(a * n, g) + np.outer(g, a * n) + D * np.outer(g, g)
         + np.outer(g, Gsum) + np.outer(Gsum, g))
    # U_new^{-T} = U^{-T} (I - lr H A H^T)^{-1}
    #            = U^{-T} - (U^{-T} H) (H^T H - A^{-1}/lr)^{-1} H^T          (Woodbury)
    S = H.T @ H - np.diag(1.0 / a) / lr
    UinvT_new = st.UinvT - (st.UinvT @ H) @ np.linalg.solve(S, H.T)
    U_new = st.U - lr * (st.U @ H) @ A @ H.T
    V_new = st.V - lr * G @ (UinvT_new @ H).T
    Q_new = st.Q - lr * (H @ grad.T + grad @ H.T) + lr * lr * (H @ N) @ H.T
    c_new = st.c - lr * H @ (a * (H.T @ st.c) + g)
    s_new = st.s - lr * H @ (a * n + D * g + Gsum)
    st.U, st.UinvT, st.V, st.Q, st.c, st.s = U_new, UinvT_new, V_new, Q_new, c_new, s_new
    return grad


def minibatch_step(st: FactoredState, H_rows, idx, val, lr: float):
    """Squared error over a minibatch, applied in place to `st`.

    Loss (eq. L, one example per column): L_i = h_i^T Q h_i - 2 h_i^T (W^T y_i)
    + y_i^T y_i; the minibatch loss is their sum (the trace of the m x m matrix
    whose diagonal they are).  dL/dO = 2 (W H - Y): a_i = 2, G = -2 Y.
    Returns (loss[m], grad_H[m x d]).
    """
    D = st.V.shape[0]
    H = widen(H_rows).T                      # d x m
    Y = dense_targets(D, idx, val)           # D x m, sparse in content
    QH = st.Q @ H
    WtY = st.WtG(Y)                          # W^T Y without forming W
    loss = (np.einsum("ji,ji->i", H, QH) - 2.0 * np.einsum("ji,ji->i", H, WtY)
            + np.einsum("ji,ji->i", Y, Y))
    m = H.shape[1]
    grad = _factored_update(st, H, np.full(m, 2.0), -2.0 * Y, QH, -2.0 * WtY, lr)
    return loss, grad.T.copy()


def spherical_minibatch_step(st: FactoredState, H_rows, idx, lr: float, eps: float = 1e-3):
    """Spherical softmax L_i = -log((o_c^2 + eps) / sum_j (o_j^2 + eps)), in place.

    With o = W h_i:  sum_j (o_j^2 + eps) = h_i^T Q h_i + D eps =: S_i and
    o_c = h_i^T (W^T e_c), both cheap (the section 3.6 family).  The output
    gradient is 2 o / S_i - 2 o_c e_c / (o_c^2 + eps), i.e. the (a, G) form with
    a_i = 2 / S_i and G = Y diag(beta), beta_i = -2 o_c / (o_c^2 + eps), Y the
    one-hot targets.  Pinned against the explicit definition and finite
    differences only (the paper prints no minibatch formulas for this loss).
    Returns (loss[m], grad_H[m x d]).
    """
    D = st.V.shape[0]
    H = widen(H_rows).T                                      # d x m
    Y = dense_targets(D, idx, None, one_hot=True)            # D x m
    QH = st.Q @ H
    WtY = st.WtG(Y)                                          # column i: W^T e_{c_i}
    oc = np.einsum("ji,ji->i", H, WtY)
    S = np.einsum("ji,ji->i", H, QH) + D * eps
    loss = -np.log((oc * oc + eps) / S)
    beta = -2.0 * oc / (oc * oc + eps)
    grad = _factored_update(st, H, 2.0 / S, Y * beta[None, :], QH, WtY * beta[None, :], lr)
    return loss, grad.T.copy()


def shifted_spherical_minibatch_step(st: FactoredState, H_rows, idx, lr: float,
                                     eps: float = 1e-3):
    """L_i = -log((o_c + eps)^2 / sum_j (o_j + eps)^2), in place (section 3.6).

    With u = o + eps 1 and s = W^T 1:  S_i = sum_j u_j^2 = h_i^T Q h_i
    + 2 eps s^T h_i + D eps^2 and u_c = h_i^T (W^T e_c) + eps.  The output
    gradient 2 u / S_i - 2 e_c / u_c is the form above with a_i = 2 / S_i,
    g = eps a (the all-ones direction) and G = Y diag(beta), beta_i = -2 / u_c.
    Pinned against the explicit definition only (the paper prints no minibatch
    formulas for this loss).  Returns (loss[m], grad_H[m x d]).
    """
    D = st.V.shape[0]
    H = widen(H_rows).T                                      # d x m
    Y = dense_targets(D, idx, None, one_hot=True)            # D x m
    QH = st.Q @ H
    WtY = st.WtG(Y)                                          # column i: W^T e_{c_i}
    uc = np.einsum("ji,ji->i", H, WtY) + eps
    S = np.einsum("ji,ji->i", H, QH) + 2.0 * eps * (H.T @ st.s) + D * eps * eps
    loss = -np.log(uc * uc / S)
    a = 2.0 / S
    beta = -2.0 / uc
    grad = _factored_update(st, H, a, Y * beta[None, :], QH, WtY * beta[None, :], lr, g=eps * a)
    return loss, grad.T.copy()


def sherman_morrison_inverse_T(UinvT, h, lr: float):
    """Eq. updateU-T: the inverse transpose of U (I - 2 lr h h^T) from that of U,
    U^{-T} + 2 lr / (1 - 2 lr ||h||^2) (U^{-T} h) h^T."""
    h = widen(h)
    return UinvT + (2.0 * lr / (1.0 - 2.0 * lr * (h @ h))) * np.outer(UinvT @ h, h)


def online_step(st: FactoredState, h, y_idx, y_val, lr: float):
    """One example, squared error, applied in place.  Returns (L, grad_h).

    The loss and the gradient come from eq. L and eq. gradH (with
    z = Q h - W^T y); the state then moves by rank-one changes only:
    U by eq. updateU, U^{-T} by eq. updateU-T, V along y by eq. updateV
    (which needs the new U^{-T} times h), and Q by eq. updateQ, whose last
    term carries the example's loss L.  The state's shared row c must be zero
    (it is for this loss); s = W^T 1 is kept up to date.
    """
    if np.any(st.c):
        raise ValueError("online_step handles states with c = 0 only")
    D = st.V.shape[0]
    h = widen(h)
    y = dense_targets(D, np.asarray(y_idx).reshape(1, -1), np.asarray(y_val).reshape(1, -1))[:, 0]
    Qh = st.Q @ h
    Wty = st.U.T @ (st.V.T @ y)
    z = Qh - Wty
    L = h @ Qh - 2.0 * (h @ Wty) + y @ y
    grad_h = 2.0 * z
    UinvT_new = sherman_morrison_inverse_T(st.UinvT, h, lr)
    st.V = st.V + 2.0 * lr * np.outer(y, UinvT_new @ h)
    st.U = st.U - 2.0 * lr * np.outer(st.U @ h, h)
    st.UinvT = UinvT_new
    st.Q = st.Q - 2.0 * lr * (np.outer(h, z) + np.outer(z, h)) + 4.0 * lr * lr * L * np.outer(h, h)
    st.s = st.s - 2.0 * lr * (st.s @ h - np.sum(y)) * h   # s - lr h (dL/do)^T 1
    return L, grad_h


def pristine_restore(st: FactoredState) -> None:
    """Appendix C: V <- V U, U <- I, U^{-T} <- I.  W and Q are unchanged."""
    d = st.U.shape[0]
    st.V = st.V @ st.U
    st.U = np.eye(d)
    st.UinvT = np.eye(d)
