"""The paper's factored algorithm, literally, in fp64 (test infrastructure only).

TEST INFRASTRUCTURE ONLY (see the package docstring).

W is never stored: it is V U (D x d times d x d, section 3.2), and the side
matrices Q = W^T W and U^{-T} are kept up to date (section 3.3).  This module
exists to check the paper's algebra against the explicit definition in
`oracle.explicit`: after every step V U must equal the explicitly updated W,
Q must equal W^T W and U (U^{-T})^T must be the identity.

Functions
  FactoredState.from_initial  Appendix A initialisation (V = W0, U = I, U^{-T} = I,
                              Q = V^T V), generalised to any invertible U0.
  minibatch_step              Appendix A, steps 1-10, squared error, in the paper's order.
  online_step                 Algorithm 1 (one example, Sherman-Morrison update of U^{-T}).
  sherman_morrison_inverse_T  equation (updateU-T) on its own.
  spherical_minibatch_step    minibatch form for the spherical softmax, derived here
                              (the paper gives no minibatch formulas for section 3.6).
  pristine_restore            Appendix C: V <- V U, U <- I, U^{-T} <- I.
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

    @classmethod
    def from_initial(cls, V0, U0=None) -> "FactoredState":
        """Appendix A initialisation.  With U0 = I this is V = W0, Q = V^T V,
        U = U^{-T} = I; a general invertible U0 gives W0 = V0 U0."""
        V = widen(V0)
        d = V.shape[1]
        U = np.eye(d) if U0 is None else widen(U0)
        W = V @ U
        return cls(V=V, U=U, UinvT=np.linalg.inv(U).T, Q=W.T @ W)

    def W(self) -> np.ndarray:
        return self.V @ self.U


def minibatch_step(st: FactoredState, H_rows, idx, val, lr: float):
    """Appendix A, steps 1-10 (squared error), applied in place to `st`.

    Returns (loss[m] = diag M, grad_H[m x d]).  The sum of loss is L = Tr M.
    """
    D = st.V.shape[0]
    H = widen(H_rows).T                      # d x m
    m = H.shape[1]
    Y = dense_targets(D, idx, val)           # D x m, sparse in content
    Hhat = st.Q @ H                                          # 1
    Yhat = st.U.T @ (st.V.T @ Y)                             # 2
    Zhat = Hhat - Yhat                                       # 3
    grad_H = 2.0 * Zhat                                      # 4
    M = H.T @ Zhat - Yhat.T @ H + Y.T @ Y                    # 5
    loss = np.diag(M).copy()                                 # 6 (L = Tr M)
    U_new = st.U - 2.0 * lr * (st.U @ H) @ H.T               # 7
    S = H.T @ H - np.eye(m) / (2.0 * lr)
    UinvT_new = st.UinvT - (st.UinvT @ H) @ np.linalg.solve(S, H.T)   # 8 (Woodbury)
    V_new = st.V + 2.0 * lr * Y @ (UinvT_new @ H).T          # 9
    Q_new = (st.Q - 2.0 * lr * (H @ Zhat.T + Zhat @ H.T)
             + 4.0 * lr * lr * (H @ M) @ H.T)                # 10
    st.U, st.UinvT, st.V, st.Q = U_new, UinvT_new, V_new, Q_new
    return loss, grad_H.T.copy()


def sherman_morrison_inverse_T(UinvT, h, lr: float):
    """Equation (updateU-T): U_new^{-T} = U^{-T} + 2 lr / (1 - 2 lr ||h||^2) (U^{-T} h) h^T."""
    h = widen(h)
    return UinvT + (2.0 * lr / (1.0 - 2.0 * lr * (h @ h))) * np.outer(UinvT @ h, h)


def online_step(st: FactoredState, h, y_idx, y_val, lr: float):
    """Algorithm 1 (one example, squared error), applied in place.  Returns (L, grad_h)."""
    D = st.V.shape[0]
    h = widen(h)
    y = dense_targets(D, np.asarray(y_idx).reshape(1, -1), np.asarray(y_val).reshape(1, -1))[:, 0]
    hhat = st.Q @ h                                          # 1
    yhat = st.U.T @ (st.V.T @ y)                             # 2
    zhat = hhat - yhat                                       # 3
    grad_h = 2.0 * zhat                                      # 4
    L = h @ hhat - 2.0 * (h @ yhat) + y @ y                  # 5
    U_new = st.U - 2.0 * lr * np.outer(st.U @ h, h)          # 6
    UinvT_new = sherman_morrison_inverse_T(st.UinvT, h, lr)  # 7
    V_new = st.V + 2.0 * lr * np.outer(y, UinvT_new @ h)     # 8
    Q_new = (st.Q - 2.0 * lr * (np.outer(h, zhat) + np.outer(zhat, h))
             + 4.0 * lr * lr * L * np.outer(h, h))           # 9
    st.U, st.UinvT, st.V, st.Q = U_new, UinvT_new, V_new, Q_new
    return L, grad_h


def spherical_minibatch_step(st: FactoredState, H_rows, idx, lr: float, eps: float = 1e-3):
    """Factored minibatch step for L_i = -log((o_c^2 + eps) / sum_j (o_j^2 + eps)).

    Derived here, following the structure of Appendix A (the paper lists the
    loss family in section 3.6 but gives no minibatch formulas).  Write the
    output gradient of the minibatch as  dL/dO = W H A + G,  with
    A = diag(a_i), a_i = 2 / S_i, S_i = h_i^T Q h_i + D eps (= sum_j (o_j^2 + eps)),
    and G = Y diag(beta_i) sparse on the targets, beta_i = -2 o_c / (o_c^2 + eps),
    o_c = h_i^T (W^T e_c).  Then W_new = W - lr (W H A + G) H^T and, exactly as in
    Appendix A:
        U_new      = U - lr (U H) A H^T
        U_new^{-T} = U^{-T} - (U^{-T} H) S_w^{-1} H^T,  S_w = H^T H - A^{-1} / lr   (Woodbury)
        V_new      = V - lr G (U_new^{-T} H)^T
        Q_new      = Q - lr (H grad_H^T + grad_H H^T) + lr^2 H N H^T
    with grad_H = Q H A + W^T G and N = (dL/dO)^T (dL/dO)
       = A H^T Q H A + A H^T (W^T G) + (W^T G)^T H A + G^T G.
    Squared error is the special case a_i = 2, G = -2 Y.
    Pinned against the explicit definition and finite differences only.
    """
    D = st.V.shape[0]
    H = widen(H_rows).T                                      # d x m
    m = H.shape[1]
    Y = dense_targets(D, idx, None, one_hot=True)            # one-hot targets, D x m
    Hhat = st.Q @ H                                          # Q H
    Yhat = st.U.T @ (st.V.T @ Y)                             # W^T Y: column i = W^T e_{c_i}
    oc = np.einsum("ji,ji->i", H, Yhat)                      # o_c = h^T W^T e_c
    S = np.einsum("ji,ji->i", H, Hhat) + D * eps             # ||o||^2 + D eps
    loss = -np.log((oc * oc + eps) / S)
    a = 2.0 / S
    beta = -2.0 * oc / (oc * oc + eps)
    A = np.diag(a)
    G = Y * beta[None, :]                                    # sparse part of dL/dO
    WtG = Yhat * beta[None, :]                               # W^T G
    grad_H = Hhat @ A + WtG
    N = A @ H.T @ Hhat @ A + A @ H.T @ WtG + WtG.T @ H @ A + G.T @ G
    U_new = st.U - lr * (st.U @ H) @ A @ H.T
    Sw = H.T @ H - np.diag(1.0 / a) / lr
    UinvT_new = st.UinvT - (st.UinvT @ H) @ np.linalg.solve(Sw, H.T)
    V_new = st.V - lr * G @ (UinvT_new @ H).T
    Q_new = st.Q - lr * (H @ grad_H.T + grad_H @ H.T) + lr * lr * (H @ N) @ H.T
    st.U, st.UinvT, st.V, st.Q = U_new, UinvT_new, V_new, Q_new
    return loss, grad_H.T.copy()


def pristine_restore(st: FactoredState) -> None:
    """Appendix C: V <- V U, U <- I, U^{-T} <- I.  W and Q are unchanged."""
    d = st.U.shape[0]
    st.V = st.V @ st.U
    st.U = np.eye(d)
    st.UinvT = np.eye(d)
