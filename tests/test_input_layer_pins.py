"""Pins of oracle.input_layer (section 2.2) against brute force and the
section's own per-pair statement of the update."""
import numpy as np
import pytest

from oracle import input_layer


def _case(seed=3, D=17, d=4, m=3, K=4):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((D, d)).astype(np.float32)
    idx = rng.integers(0, D, size=(m, K)).astype(np.int32)
    idx[0, 1] = idx[0, 0]          # repeated inside an example
    idx[2, 0] = idx[1, 3]          # shared by two examples
    idx[1, 2] = -1                 # padding
    val = rng.standard_normal((m, K)).astype(np.float32)
    return W, idx, val


def test_forward_is_the_sum_of_the_selected_rows():
    W, idx, val = _case()
    A = input_layer.forward(W, idx, val)
    for i in range(idx.shape[0]):
        want = np.zeros(W.shape[1])
        for k in range(idx.shape[1]):
            if idx[i, k] >= 0:
                want += float(val[i, k]) * W[idx[i, k]].astype(np.float64)
        np.testing.assert_allclose(A[i], want, rtol=1e-15, atol=1e-15)


def test_update_is_the_per_pair_rule():
    """Section 2.2: W[u_k] <- W[u_k] - lr v_k grad_a for every pair of every
    example (the minibatch sums the examples' rank-one updates)."""
    W, idx, val = _case()
    rng = np.random.default_rng(9)
    G = rng.standard_normal((idx.shape[0], W.shape[1]))
    lr = 0.3
    got = input_layer.update(W, idx, val, G, lr)
    want = W.astype(np.float64).copy()
    for i in range(idx.shape[0]):
        for k in range(idx.shape[1]):
            if idx[i, k] >= 0:
                want[idx[i, k]] -= lr * float(val[i, k]) * G[i]
    np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-14)
    untouched = np.setdiff1d(np.arange(W.shape[0]), idx[idx >= 0])
    np.testing.assert_array_equal(got[untouched], W[untouched].astype(np.float64))


def test_gradient_of_a_linear_functional():
    """d/dW of sum(A * G) is X^T G, so one update step with lr = eps changes
    sum(A * G) by -eps ||X^T G||^2 exactly (A is linear in W)."""
    W, idx, val = _case(seed=5)
    G = np.random.default_rng(2).standard_normal((idx.shape[0], W.shape[1]))
    f0 = float(np.sum(input_layer.forward(W, idx, val) * G))
    eps = 1e-3
    W1 = input_layer.update(W, idx, val, G, eps)
    f1 = float(np.sum(input_layer.forward(W1, idx, val) * G))
    XtG = input_layer.dense_inputs(W.shape[0], idx, val).T @ G
    assert abs((f1 - f0) - (-eps * float(np.sum(XtG * XtG)))) < 1e-12


def test_bad_index_rejected():
    W, idx, val = _case()
    idx[0, 0] = W.shape[0]
    with pytest.raises(IndexError):
        input_layer.forward(W, idx, val)
