"""The sparse input layer of section 2.2 ("the easy part"), plainly, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A K-sparse input x of dimension D_in is given as (index, value) pairs: x_u = v
for each pair, 0 elsewhere (section 2.2; index -1 marks an unused pair, and an
index repeated inside one example adds its values, as for the targets).  For a
minibatch the examples are the rows of X (m x D_in, sparse):

  forward   A = X W_in               (m x d): row i = sum_k v_ik W_in[u_ik, :]
  update    W_in <- W_in - lr X^T dA  (only the rows some example refers to change)

Both are written here from the definition with a dense X; `dense_inputs`
builds X.  Pins: tests/test_input_layer_pins.py (brute-force loops on tiny
inputs, the section's per-pair update rule, untouched rows, repeated and
shared indices, the exact first-order change of a linear functional).
"""
from __future__ import annotations

import numpy as np

from .explicit import widen


def dense_inputs(D_in: int, idx, val) -> np.ndarray:
    """Dense X (m x D_in) from each example's (index, value) pairs."""
    idx = np.asarray(idx)
    m, K = idx.shape
    X = np.zeros((m, D_in), dtype=np.float64)
    for i in range(m):
        for k in range(K):
            r = int(idx[i, k])
            if r == -1:
                continue
            if r < -1 or r >= D_in:
                raise IndexError(f"input index {r} outside [-1, {D_in})")
            X[i, r] += float(val[i, k])
    return X


def forward(W_in, idx, val) -> np.ndarray:
    """A = X W_in: the first hidden layer's pre-activations of the minibatch."""
    W = widen(W_in)
    return dense_inputs(W.shape[0], idx, val) @ W


def update(W_in, idx, val, grad_A, lr: float) -> np.ndarray:
    """W_in - lr X^T grad_A (grad_A = dL/dA, m x d); returns the new W_in."""
    W = widen(W_in)
    X = dense_inputs(W.shape[0], idx, val)
    return W - lr * (X.T @ widen(grad_A))
