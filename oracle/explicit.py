"""Explicit-W fp64 reference: the plain definition of the output-layer step.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Notation follows the paper (section 2.1): W is the D x d output weight matrix,
h a d-dimensional last hidden representation, o = W h the D-dimensional output
and y the K-sparse target.  A minibatch stacks m examples as the columns of H
(d x m) and Y (D x m) (Appendix A).  The arrays handed in are row-major with
one example per row (H_rows = H^T), which is the same memory as the paper's
column layout; this module transposes them back to the paper's notation.

Every function widens its fp32 inputs to fp64 exactly and computes the naive
O(Dd)-per-example quantities the factored method must reproduce exactly
(section 3, and the experimental check of section 4 that VU equals the
explicitly trained W).

Readings of the paper taken here:
  * learning rate: W <- W - lr * dL/dW with L the SUM of the per-example
    losses of the minibatch, so squared error uses 2*lr (section 3.2 and the
    minibatch algorithm of Appendix A, whose L = Tr M is a sum);
  * a target is a list of (index, value) pairs (section 2.1); index -1 marks an
    unused slot and a repeated index adds its values;
  * spherical softmax: L_i = -log((o_c^2 + eps) / sum_k (o_k^2 + eps)) with one
    target class c per example, eps = 1e-3; this is a member of the family of
    section 3.6 (a function of o_c and ||o||^2 only);
  * shifted spherical softmax: the form section 3.6 prints,
    L_i = -log((o_c + eps)^2 / sum_k (o_k + eps)^2), one class per example.  It
    also needs sum_k o_k, so it lies just outside the family as the paper states
    it; the factored oracle carries the extra terms (oracle.factored).
"""
from __future__ import annotations

from typing import Iterable, Iterator, Tuple

import numpy as np


def widen(x) -> np.ndarray:
    """fp32 (or any) array -> fp64 copy; exact for fp32 inputs."""
    return np.array(x, dtype=np.float64, copy=True)


def dense_targets(D: int, idx: np.ndarray, val: np.ndarray, one_hot: bool = False) -> np.ndarray:
    """Dense Y (D x m) from the (index, value) pairs of each example (section 2.1).

    Column i is example i's target vector: y[idx[i,k]] += val[i,k] for every
    slot k with idx[i,k] >= 0 (a repeated index adds up).  With one_hot the
    value of each pair is taken as 1 (classification targets).
    Raises IndexError for an index outside [-1, D).
    """
    idx = np.asarray(idx)
    m, K = idx.shape
    Y = np.zeros((D, m), dtype=np.float64)
    for i in range(m):
        for k in range(K):
            r = int(idx[i, k])
            if r == -1:
                continue
            if r < -1 or r >= D:
                raise IndexError(f"target index {r} outside [-1, {D})")
            Y[r, i] += 1.0 if one_hot else float(val[i, k])
    return Y


def touched_rows(idx: np.ndarray) -> np.ndarray:
    """Sorted distinct target indices of a minibatch: the rows of W that the
    sparse part of the update visits (section 3.2, the O(Kd) update of V)."""
    idx = np.asarray(idx).ravel()
    return np.unique(idx[idx >= 0]).astype(np.int64)


def target_gram(D: int, idx: np.ndarray, val: np.ndarray, one_hot: bool = False) -> np.ndarray:
    """Y^T Y (m x m), the target term of M in the minibatch algorithm (Appendix A, step 5)."""
    Y = dense_targets(D, idx, val, one_hot)
    return Y.T @ Y


def squared_error_step(W, H_rows, idx, val, lr: float):
    """One minibatch step of the naive linear output + squared error layer.

    Section 2.3 / 3.1 / 3.2: o = W h, L = ||o - y||^2, grad_h = 2 W^T (o - y),
    W_new = W - 2 lr (o - y) h^T, summed over the m examples.

    Returns (loss[m], grad_H[m x d] (row i = grad wrt h_i), W_new[D x d]), fp64.
    """
    W = widen(W)
    D = W.shape[0]
    H = widen(H_rows).T                     # d x m, columns are examples
    Y = dense_targets(D, idx, val)          # D x m
    O = W @ H                               # outputs, D x m   -- O(Dd) per example
    R = O - Y                               # residuals
    loss = np.einsum("jm,jm->m", R, R)      # ||o_i - y_i||^2
    grad_H = 2.0 * (W.T @ R)                # d x m
    grad_W = 2.0 * (R @ H.T)                # dL/dW = sum_i 2 (o_i - y_i) h_i^T
    W_new = W - lr * grad_W
    return loss, grad_H.T.copy(), W_new


def spherical_softmax_step(W, H_rows, idx, lr: float, eps: float = 1e-3):
    """One minibatch step of the naive spherical-softmax output layer.

    Section 3.6 loss family, in the form
        L_i = -log((o_c^2 + eps) / sum_j (o_j^2 + eps)),   o = W h_i,
    with c = idx[i, 0] the target class.  Its output gradient is
        dL_i/do = 2 o / S_i - 2 o_c e_c / (o_c^2 + eps),   S_i = sum_j (o_j^2 + eps),
    back-propagated as grad_h = W^T dL/do and applied as W_new = W - lr dL/dW.

    Returns (loss[m], grad_H[m x d], W_new[D x d]), fp64.
    """
    W = widen(W)
    D = W.shape[0]
    H = widen(H_rows).T                     # d x m
    m = H.shape[1]
    c = np.asarray(idx)[:, 0].astype(np.int64)
    if np.any(c < 0) or np.any(c >= D):
        raise IndexError("spherical softmax needs one target class in [0, D) per example")
    O = W @ H                               # D x m
    cols = np.arange(m)
    S = np.sum(O * O + eps, axis=0)         # sum_j (o_j^2 + eps)
    oc = O[c, cols]
    loss = -np.log((oc * oc + eps) / S)
    G = 2.0 * O / S                         # dL/dO, dense part
    G[c, cols] -= 2.0 * oc / (oc * oc + eps)  # sparse part at the target classes
    grad_H = W.T @ G
    W_new = W - lr * (G @ H.T)
    return loss, grad_H.T.copy(), W_new


def shifted_spherical_step(W, H_rows, idx, lr: float, eps: float = 1e-3):
    """One minibatch step of the spherical softmax in the form section 3.6 prints.

        L_i = -log((o_c + eps)^2 / sum_j (o_j + eps)^2),   o = W h_i,
    c = idx[i, 0] the target class.  With u = o + eps (every output shifted by
    eps) and S_i = sum_j u_j^2, the output gradient is
        dL_i/do = 2 u / S_i - 2 e_c / u_c,
    back-propagated as grad_h = W^T dL/do and applied as W_new = W - lr dL/dW.

    Returns (loss[m], grad_H[m x d], W_new[D x d]), fp64.
    """
    W = widen(W)
    D = W.shape[0]
    H = widen(H_rows).T                     # d x m
    m = H.shape[1]
    c = np.asarray(idx)[:, 0].astype(np.int64)
    if np.any(c < 0) or np.any(c >= D):
        raise IndexError("spherical softmax needs one target class in [0, D) per example")
    Uo = W @ H + eps                        # D x m, the shifted outputs
    cols = np.arange(m)
    S = np.sum(Uo * Uo, axis=0)
    uc = Uo[c, cols]
    loss = -np.log(uc * uc / S)
    G = 2.0 * Uo / S
    G[c, cols] -= 2.0 / uc
    grad_H = W.T @ G
    W_new = W - lr * (G @ H.T)
    return loss, grad_H.T.copy(), W_new


def term_scales(W, H_rows, idx, val, loss, grad_H, loss_kind: str = "squared",
                eps: float = 1e-3):
    """Per-example magnitudes of the terms whose sums give L_i and grad_h_i.

    A method that never forms o = W h evaluates the loss and the gradient as
    sums of a few terms (eq. L and eq. gradH of section 3.1; the section 3.6
    family for the spherical softmax):
      squared    L_i = h^T Q h - 2 h^T W^T y + y^T y,   grad = 2 W^T W h - 2 W^T y;
      spherical  L_i = log S_i - log(o_c^2 + eps),      grad = (2/S_i) W^T W h + b_i W^T e_c,
                 b_i = -2 o_c / (o_c^2 + eps), S_i = sum_j (o_j^2 + eps);
      shifted    L_i = log S_i - log(u_c^2),  grad = (2/S_i)(W^T W h + eps s) + b_i W^T e_c,
                 u = o + eps, b_i = -2 / u_c, s = W^T 1, and
                 S_i = h^T W^T W h + 2 eps s^T h + D eps^2 a sum of three terms.
    The rounding error of any evaluation of such a sum is bounded by a multiple
    of the sum of the terms' magnitudes, which can exceed |L_i| or ||grad_i||
    many times when the terms cancel.  For the spherical softmax the scales
    also carry the sensitivity of L_i and of the class term of grad_i to o_c,
    a sum of terms of total size |w_c| |h_i| (w_c the class row of W).  Returns (loss_scale[m], grad_scale[m]):
    sum of |term| for L_i and sum of ||term|| for grad_h_i, at W (the weights
    the step starts from), loss and grad_H (the step's exact loss[m] and
    gradient, m x d).  Costs O(m K d): the dense terms come from grad_H and
    the sparse ones, log S_i from L_i.
    """
    W = widen(W)
    H = widen(H_rows)                        # m x d, rows are examples
    g = widen(grad_H)
    idx = np.asarray(idx)
    m = H.shape[0]
    loss_scale = np.zeros(m)
    grad_scale = np.zeros(m)
    s1 = W.sum(axis=0) if loss_kind == "spherical_shifted" else None
    for i in range(m):
        if loss_kind == "squared":
            wty = np.zeros(W.shape[1])
            yv = {}
            for k in range(idx.shape[1]):
                r = int(idx[i, k])
                if r < 0:
                    continue
                yv[r] = yv.get(r, 0.0) + float(val[i, k])
            for r, v in yv.items():
                wty += v * W[r]
            yy = sum(v * v for v in yv.values())
            wtwh = 0.5 * g[i] + wty                   # W^T W h from grad = 2 (W^T W h - W^T y)
            loss_scale[i] = abs(H[i] @ wtwh) + 2.0 * abs(H[i] @ wty) + yy
            grad_scale[i] = 2.0 * np.linalg.norm(wtwh) + 2.0 * np.linalg.norm(wty)
        elif loss_kind == "spherical":
            c = int(idx[i, 0])
            wc = W[c]
            oc = float(wc @ H[i])
            b = -2.0 * oc / (oc * oc + eps)
            t = b * wc
            lo = np.log(oc * oc + eps)
            # o_c = w_c . h is itself a sum, of terms of total size |w_c| |h|; a
            # change of o_c moves L_i by b dO_c and the class term of the
            # gradient by b'(o_c) dO_c w_c, b' = 2 (o_c^2 - eps) / (o_c^2 + eps)^2,
            # up to 2 / eps in size near o_c = 0
            doc = float(np.linalg.norm(wc) * np.linalg.norm(H[i]))
            db = 2.0 * (oc * oc - eps) / (oc * oc + eps) ** 2
            loss_scale[i] = abs(lo) + abs(float(loss[i]) + lo) + abs(b) * doc
            grad_scale[i] = (np.linalg.norm(g[i] - t) + np.linalg.norm(t)
                             + abs(db) * doc * np.linalg.norm(wc))
        elif loss_kind == "spherical_shifted":
            c = int(idx[i, 0])
            wc = W[c]
            uc = float(wc @ H[i]) + eps
            b = -2.0 / uc
            t = b * wc
            S = uc * uc * np.exp(float(loss[i]))          # L_i = log S_i - log u_c^2
            sterm = (2.0 * eps / S) * s1                  # (2/S) eps s
            qterm = g[i] - t - sterm                      # (2/S) W^T W h
            hn = float(np.linalg.norm(H[i]))
            # S_i is formed from terms of total size s_terms; its relative error
            # moves log S_i and scales the dense part of the gradient
            s_terms = 0.5 * S * abs(float(H[i] @ qterm)) + 2.0 * eps * np.linalg.norm(s1) * hn \
                + W.shape[0] * eps * eps
            doc = float(np.linalg.norm(wc)) * hn
            db = 2.0 / (uc * uc)                          # slope of b in o_c
            lu = np.log(uc * uc)
            loss_scale[i] = abs(lu) + abs(float(loss[i]) + lu) + abs(b) * doc + s_terms / S
            grad_scale[i] = ((np.linalg.norm(qterm) + np.linalg.norm(sterm)) * (1.0 + s_terms / S)
                             + np.linalg.norm(t) + db * doc * np.linalg.norm(wc))
        else:
            raise ValueError(f"unknown loss {loss_kind!r}")
    return loss_scale, grad_scale


def step_fp32(W, H_rows, idx, val, lr: float, loss_kind: str = "squared", eps: float = 1e-3):
    """The same definition as `step`, evaluated in float32 arithmetic.

    Not a reference: a yardstick.  Its distance from the fp64 trajectory shows
    how closely any fp32 evaluation of the method can follow that trajectory
    (the spherical softmax amplifies rounding through -2 o_c / (o_c^2 + eps),
    whose slope at small o_c is up to 2 / eps).  Returns (loss, grad_H, W_new)
    as float32 arrays.
    """
    f = np.float32
    W = np.asarray(W, dtype=f)
    D = W.shape[0]
    H = np.asarray(H_rows, dtype=f).T
    m = H.shape[1]
    O = W @ H
    if loss_kind == "squared":
        Y = dense_targets(D, idx, val).astype(f)
        R = O - Y
        loss = np.einsum("jm,jm->m", R, R)
        G = f(2.0) * R
    elif loss_kind == "spherical":
        c = np.asarray(idx)[:, 0].astype(np.int64)
        cols = np.arange(m)
        S = np.sum(O * O + f(eps), axis=0, dtype=f)
        oc = O[c, cols]
        loss = -np.log((oc * oc + f(eps)) / S)
        G = f(2.0) * O / S
        G[c, cols] -= f(2.0) * oc / (oc * oc + f(eps))
    elif loss_kind == "spherical_shifted":
        c = np.asarray(idx)[:, 0].astype(np.int64)
        cols = np.arange(m)
        Uo = O + f(eps)
        S = np.sum(Uo * Uo, axis=0, dtype=f)
        uc = Uo[c, cols]
        loss = -np.log(uc * uc / S)
        G = f(2.0) * Uo / S
        G[c, cols] -= f(2.0) / uc
    else:
        raise ValueError(f"unknown loss {loss_kind!r}")
    grad = (W.T @ G).T.copy()
    W_new = W - f(lr) * (G @ H.T)
    return loss, grad, W_new


def step(W, H_rows, idx, val, lr: float, loss_kind: str = "squared", eps: float = 1e-3):
    """Dispatch on the loss: 'squared', 'spherical' or 'spherical_shifted'."""
    if loss_kind == "squared":
        return squared_error_step(W, H_rows, idx, val, lr)
    if loss_kind == "spherical":
        return spherical_softmax_step(W, H_rows, idx, lr, eps)
    if loss_kind == "spherical_shifted":
        return shifted_spherical_step(W, H_rows, idx, lr, eps)
    raise ValueError(f"unknown loss {loss_kind!r}")


def trajectory(
    W0, batches: Iterable[Tuple[np.ndarray, np.ndarray, np.ndarray]], lr: float,
    loss_kind: str = "squared", eps: float = 1e-3,
) -> Iterator[Tuple[np.ndarray, np.ndarray, np.ndarray]]:
    """Run consecutive steps from W0; yields (loss, grad_H, W_after) per step."""
    W = widen(W0)
    for H, idx, val in batches:
        loss, grad_H, W = step(W, H, idx, val, lr, loss_kind, eps)
        yield loss, grad_H, W
