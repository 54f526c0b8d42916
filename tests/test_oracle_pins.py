"""Pins of the fp64 oracle against facts other than itself.

Each test fixes part of `oracle/` by something the paper or mathematics
determines: a hand-derived worked example, closed forms of special cases,
finite differences of the loss, the paper's identities (eq. L, eq. gradH, the
exactness proof of section 3.2, the Q bookkeeping of Appendix B, Woodbury vs
Sherman-Morrison), brute force on tiny inputs.  The last test plants plausible
mistakes in the oracle and checks that these pins catch every one.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import explicit, factored
from synth import Workload, WorkloadConfig

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def _tiny(loss="squared", seed=7, D=23, d=5, m=4, K=3, **kw):
    cfg = WorkloadConfig(
        name="tiny", D=D, d=d, m=m, K=K, loss=loss, lr=0.05, steps=5,
        idx_dist="uniform", distinct=False, val_dist="normal", h_scale=0.7,
        v_bound=0.5, entropy=seed, **kw,
    )
    return Workload(cfg)


# ------------------------------------------------------------ worked examples
def check_worked_squared(step_fn):
    g = _golden()["squared"]
    loss, grad, W_new = step_fn(
        np.array(g["W"], np.float32), np.array(g["H"], np.float32),
        np.array(g["idx"], np.int32), np.array(g["val"], np.float32), g["lr"],
    )
    np.testing.assert_array_equal(loss, np.array(g["loss"], np.float64))
    np.testing.assert_array_equal(grad, np.array(g["grad_H"], np.float64))
    np.testing.assert_array_equal(W_new, np.array(g["W_new"], np.float64))


def test_worked_example_squared():
    check_worked_squared(explicit.squared_error_step)
    g = _golden()["squared"]
    idx = np.array(g["idx"], np.int32)
    val = np.array(g["val"], np.float32)
    np.testing.assert_array_equal(explicit.touched_rows(idx), g["touched_rows"])
    np.testing.assert_array_equal(explicit.target_gram(3, idx, val), np.array(g["YtY"], float))


def test_worked_example_spherical():
    g = _golden()["spherical"]
    loss, grad, W_new = explicit.spherical_softmax_step(
        np.array(g["W"], np.float32), np.array(g["H"], np.float32),
        np.array(g["idx"], np.int32), g["lr"], g["eps"],
    )
    S = Fraction(*g["S_rational"])
    num = Fraction(*g["oc2_plus_eps_rational"])
    assert abs(loss[0] - math.log(S / num)) < 1e-14
    d0 = Fraction(*g["dLdo_rational"][0])
    d1 = Fraction(*g["dLdo_rational"][1])
    d2 = sum(Fraction(*p) for p in g["dLdo_rational"][2])
    want = np.array([float(d0 + d2), float(d1 + d2)])  # W^T dL/do for W = [[1,0],[0,1],[1,1]]
    np.testing.assert_allclose(grad[0], want, rtol=1e-14, atol=0)
    h = np.array(g["H"][0], float)
    dLdo = np.array([float(d0), float(d1), float(d2)])
    np.testing.assert_allclose(W_new, np.array(g["W"], float) - g["lr"] * np.outer(dLdo, h),
                               rtol=1e-14, atol=1e-15)


def test_worked_example_shifted():
    """The hand-derived shifted example (section 3.6 as printed), in rationals."""
    g = _golden()["shifted"]
    loss, grad, W_new = explicit.shifted_spherical_step(
        np.array(g["W"], np.float32), np.array(g["H"], np.float32),
        np.array(g["idx"], np.int32), g["lr"], g["eps"],
    )
    S = Fraction(*g["S_rational"])
    uc2 = Fraction(*g["uc2_rational"])
    assert abs(loss[0] - math.log(S / uc2)) < 1e-14
    want = np.array([float(Fraction(*q)) for q in g["grad_rational"]])
    np.testing.assert_allclose(grad[0], want, rtol=1e-14, atol=0)
    h = np.array(g["H"][0], float)
    dLdo = np.array([float(Fraction(*q)) for q in g["dLdo_rational"]])
    np.testing.assert_allclose(W_new, np.array(g["W"], float) - g["lr"] * np.outer(dLdo, h),
                               rtol=1e-14, atol=1e-15)


# ---------------------------------------------------------------- closed forms
def test_identity_weights_closed_form():
    """D = d, W = I: o = h, so L = ||h - y||^2 and grad_h = 2 (h - y)."""
    d, m = 6, 3
    rng = np.random.default_rng(3)
    H = rng.standard_normal((m, d)).astype(np.float32)
    idx = np.array([[0, 5], [2, -1], [4, 4]], np.int32)
    val = rng.standard_normal((m, 2)).astype(np.float32)
    Yrows = np.zeros((m, d))
    for i in range(m):
        for k in range(2):
            if idx[i, k] >= 0:
                Yrows[i, idx[i, k]] += float(val[i, k])
    lr = 0.25
    loss, grad, W_new = explicit.squared_error_step(np.eye(d, dtype=np.float32), H, idx, val, lr)
    R = H.astype(float) - Yrows
    np.testing.assert_allclose(loss, (R * R).sum(1), rtol=1e-14)
    np.testing.assert_allclose(grad, 2 * R, rtol=1e-14)
    np.testing.assert_allclose(W_new, np.eye(d) - 2 * lr * R.T @ H.astype(float), rtol=1e-14, atol=1e-15)


def test_zero_weights_spherical_is_uniform():
    """W = 0: every output is 0, every class has probability eps / (D eps) = 1/D,
    so L_i = log D exactly and the gradient vanishes."""
    D, d, m = 17, 4, 3
    H = np.random.default_rng(0).standard_normal((m, d)).astype(np.float32)
    idx = np.array([[3], [0], [16]], np.int32)
    loss, grad, W_new = explicit.spherical_softmax_step(np.zeros((D, d), np.float32), H, idx, 0.1)
    np.testing.assert_allclose(loss, np.full(m, math.log(D)), rtol=1e-15)
    assert np.all(grad == 0) and np.all(W_new == 0)


def test_lr_zero_leaves_W_unchanged():
    wl = _tiny()
    W = wl.init_V()
    H, idx, val = wl.batch(0)
    for fn in (lambda: explicit.squared_error_step(W, H, idx, val, 0.0),
               lambda: explicit.spherical_softmax_step(W, H, np.abs(idx[:, :1]), 0.0)):
        _, _, W_new = fn()
        np.testing.assert_array_equal(W_new, W.astype(np.float64))


# ------------------------------------------------------- finite differences
def _total_loss(step_fn, W, H, idx, val):
    loss, _, _ = step_fn(W, H, idx, val, 0.0)
    return float(np.sum(loss))


def check_fd_grad_h(step_fn, idx_for=lambda idx: idx, eps_fd=1e-6, tol=1e-6):
    wl = _tiny(seed=11)
    W = wl.init_V().astype(np.float64)
    H, idx, val = wl.batch(0)
    idx = idx_for(idx)
    H = H.astype(np.float64)
    _, grad, _ = step_fn(W, H, idx, val, 0.0)
    fd = np.zeros_like(H)
    for i in range(H.shape[0]):
        for j in range(H.shape[1]):
            Hp = H.copy(); Hp[i, j] += eps_fd
            Hm = H.copy(); Hm[i, j] -= eps_fd
            fd[i, j] = (_total_loss(step_fn, W, Hp, idx, val) - _total_loss(step_fn, W, Hm, idx, val)) / (2 * eps_fd)
    assert _rel(grad, fd) < tol, _rel(grad, fd)


def check_fd_update_W(step_fn, idx_for=lambda idx: idx, eps_fd=1e-6, tol=1e-6, lr=0.01):
    """W_new = W - lr dL/dW, with dL/dW from central differences of the loss."""
    wl = _tiny(seed=13, D=9, d=3, m=3, K=2)
    W = wl.init_V().astype(np.float64)
    H, idx, val = wl.batch(0)
    idx = idx_for(idx)
    _, _, W_new = step_fn(W, H, idx, val, lr)
    fd = np.zeros_like(W)
    for r in range(W.shape[0]):
        for j in range(W.shape[1]):
            Wp = W.copy(); Wp[r, j] += eps_fd
            Wm = W.copy(); Wm[r, j] -= eps_fd
            fd[r, j] = (_total_loss(step_fn, Wp, H, idx, val) - _total_loss(step_fn, Wm, H, idx, val)) / (2 * eps_fd)
    assert _rel((W - W_new) / lr, fd) < tol, _rel((W - W_new) / lr, fd)


def _sph(W, H, idx, val, lr):
    return explicit.spherical_softmax_step(W, H, idx, lr)


def _one_class(idx):
    return np.abs(idx[:, :1])  # a valid class per example (distinct=False draws are >= 0)


def test_fd_grad_h_squared():
    check_fd_grad_h(explicit.squared_error_step)


def test_fd_grad_h_spherical():
    check_fd_grad_h(_sph, idx_for=_one_class)


def test_fd_update_W_squared():
    check_fd_update_W(explicit.squared_error_step)


def test_fd_update_W_spherical():
    check_fd_update_W(_sph, idx_for=_one_class)


def test_spherical_probabilities_sum_to_one():
    """p_c = exp(-L) summed over every possible class c is 1 (section 3.6: normalised)."""
    D, d, m = 11, 3, 2
    rng = np.random.default_rng(5)
    W = rng.standard_normal((D, d)).astype(np.float32)
    H = rng.standard_normal((m, d)).astype(np.float32)
    tot = np.zeros(m)
    for c in range(D):
        loss, _, _ = explicit.spherical_softmax_step(W, H, np.full((m, 1), c, np.int32), 0.0)
        p = np.exp(-loss)
        assert np.all(p > 0) and np.all(p <= 1)
        tot += p
    np.testing.assert_allclose(tot, np.ones(m), rtol=1e-13)


# ------------------------------------- shifted spherical softmax (section 3.6)
def _shift(W, H, idx, val, lr):
    return explicit.shifted_spherical_step(W, H, idx, lr)


def check_shift_zero_weights(step_fn):
    """W = 0: every shifted output is eps, so each class has probability
    eps^2 / (D eps^2) = 1/D, L_i = log D, and dL/do = (2 / (D eps)) 1 - (2 / eps) e_c:
    grad_h = W^T dL/do = 0 and W_new = -lr dL/dO H^T."""
    D, d, m, eps, lr = 13, 4, 3, 1e-3, 0.1
    H = np.random.default_rng(3).standard_normal((m, d)).astype(np.float32)
    idx = np.array([[5], [0], [5]], np.int32)
    loss, grad, W_new = step_fn(np.zeros((D, d), np.float32), H, idx, None, lr)
    np.testing.assert_allclose(loss, np.full(m, math.log(D)), rtol=1e-14)
    np.testing.assert_allclose(grad, np.zeros((m, d)), atol=1e-12)
    Hd = H.astype(np.float64)
    want = np.tile(-lr * (2.0 / (D * eps)) * Hd.sum(axis=0), (D, 1))
    want[5] += lr * (2.0 / eps) * (Hd[0] + Hd[2])
    want[0] += lr * (2.0 / eps) * Hd[1]
    np.testing.assert_allclose(W_new, want, rtol=1e-12, atol=1e-12)


def check_shift_sums_to_one(step_fn):
    """p_c = exp(-L) = (o_c + eps)^2 / sum_j (o_j + eps)^2 over all classes c sums to 1."""
    D, d, m = 11, 3, 2
    rng = np.random.default_rng(6)
    W = rng.standard_normal((D, d)).astype(np.float32)
    H = rng.standard_normal((m, d)).astype(np.float32)
    tot = np.zeros(m)
    for c in range(D):
        loss, _, _ = step_fn(W, H, np.full((m, 1), c, np.int32), None, 0.0)
        p = np.exp(-loss)
        assert np.all(p > 0) and np.all(p <= 1)
        tot += p
    np.testing.assert_allclose(tot, np.ones(m), rtol=1e-13)


def check_shift_fd_grad_h(step_fn):
    check_fd_grad_h(step_fn, idx_for=_one_class)


def check_shift_fd_update_W(step_fn):
    check_fd_update_W(step_fn, idx_for=_one_class)


def test_shifted_zero_weights_closed_form():
    check_shift_zero_weights(_shift)


def test_shifted_probabilities_sum_to_one():
    check_shift_sums_to_one(_shift)


def test_fd_grad_h_shifted():
    check_shift_fd_grad_h(_shift)


def test_fd_update_W_shifted():
    check_shift_fd_update_W(_shift)


def test_shifted_is_unshifted_with_a_constant_input():
    """Appending a constant input eps to h and a column of ones to W turns o + eps
    into the plain output o' = [W 1] [h; eps], and the shifted loss into the
    spherical softmax of o' at eps = 0 (a different function, pinned on its own):
    equal losses, grad_h the first d components, W_new the first d columns."""
    wl = _tiny(seed=37, D=19, d=4, m=5, K=1)
    W = wl.init_V().astype(np.float64)
    H, idx, _ = wl.batch(0)
    idx = _one_class(idx)
    eps, lr = 0.3, 0.05   # a large eps, so that dropping it anywhere shows
    L1, g1, W1 = explicit.shifted_spherical_step(W, H, idx, lr, eps)
    Wa = np.hstack([W, np.ones((W.shape[0], 1))])
    Ha = np.hstack([H.astype(np.float64), np.full((H.shape[0], 1), eps)])
    L2, g2, W2 = explicit.spherical_softmax_step(Wa, Ha, idx, lr, 0.0)
    np.testing.assert_allclose(L1, L2, rtol=1e-13)
    np.testing.assert_allclose(g1, g2[:, :-1], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(W1, W2[:, :-1], rtol=1e-12, atol=1e-13)


def _shift_mutants():
    """Plausible mistakes in the shifted loss, planted in the oracle's outputs."""
    eps = 1e-3

    def unshifted_form(W, H, idx, val, lr):       # (o_c^2 + eps) / sum (o_j^2 + eps)
        return explicit.spherical_softmax_step(W, H, idx, lr, eps)

    def ones_direction_dropped(W, H, idx, val, lr):  # W update without the eps 1 a^T term
        loss, g, Wn = _shift(W, H, idx, val, lr)
        Wd = np.asarray(W, float)
        Hd = np.asarray(H, float)
        Uo = Wd @ Hd.T + eps
        a = 2.0 / np.sum(Uo * Uo, axis=0)
        return loss, g, Wn - lr * eps * np.outer(np.ones(Wd.shape[0]), a @ Hd)

    def grad_without_s(W, H, idx, val, lr):        # grad_h missing (2 eps / S) W^T 1
        loss, g, Wn = _shift(W, H, idx, val, lr)
        Wd = np.asarray(W, float)
        Uo = Wd @ np.asarray(H, float).T + eps
        a = 2.0 / np.sum(Uo * Uo, axis=0)
        return loss, g - eps * np.outer(a, Wd.sum(axis=0)), Wn

    def class_term_squared(W, H, idx, val, lr):    # -2 u_c / u_c^2 written as -2 u_c
        Wd = np.asarray(W, float)
        Hd = np.asarray(H, float)
        loss, g, Wn = _shift(W, H, idx, val, lr)
        c = np.asarray(idx)[:, 0]
        uc = np.einsum("id,id->i", Wd[c], Hd) + eps
        dG = 2.0 / uc - 2.0 * uc                   # replaces -2/u_c by -2 u_c
        g2 = g + dG[:, None] * Wd[c]
        Wn2 = Wn.copy()
        for i in range(len(c)):
            Wn2[c[i]] -= lr * dG[i] * Hd[i]
        return loss, g2, Wn2

    return [unshifted_form, ones_direction_dropped, grad_without_s, class_term_squared]


def test_shifted_planted_mistakes_are_caught():
    pins = [check_shift_zero_weights, check_shift_sums_to_one, check_shift_fd_grad_h,
            check_shift_fd_update_W]
    for fn in pins:
        fn(_shift)
    for mutant in _shift_mutants():
        caught = False
        for fn in pins:
            try:
                fn(mutant)
            except AssertionError:
                caught = True
                break
        assert caught, f"mutant {mutant.__name__} slipped through every pin"


def test_loss_and_gradient_identities():
    """eq. L and eq. gradH (section 3.1): L = h^T Q h - 2 h^T W^T y + y^T y and
    grad_h = 2 (Q h - W^T y), with Q = W^T W."""
    wl = _tiny(seed=17, pad_frac=0.2, dup_frac=0.3)
    W = wl.init_V().astype(np.float64)
    H, idx, val = wl.batch(0)
    loss, grad, _ = explicit.squared_error_step(W, H, idx, val, 0.0)
    Q = W.T @ W
    Y = np.zeros((W.shape[0], H.shape[0]))
    for i in range(H.shape[0]):
        for k in range(idx.shape[1]):
            if idx[i, k] >= 0:
                Y[idx[i, k], i] += float(val[i, k])
    for i in range(H.shape[0]):
        h = H[i].astype(float)
        yh = W.T @ Y[:, i]
        assert abs(loss[i] - (h @ Q @ h - 2 * h @ yh + Y[:, i] @ Y[:, i])) < 1e-12 * max(1, loss[i])
        np.testing.assert_allclose(grad[i], 2 * (Q @ h - yh), rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------- index handling
def test_index_handling_brute_force():
    wl = _tiny(seed=19, D=7, m=6, K=5, pad_frac=0.25, dup_frac=0.4)
    H, idx, val = wl.batch(0)
    assert (idx == -1).any()
    rows = sorted({int(r) for r in idx.ravel() if r >= 0})
    np.testing.assert_array_equal(explicit.touched_rows(idx), rows)
    Y = explicit.dense_targets(7, idx, val)
    ycols = []
    for i in range(idx.shape[0]):
        col = {}
        for k in range(idx.shape[1]):
            r = int(idx[i, k])
            if r >= 0:
                col[r] = col.get(r, 0.0) + float(val[i, k])
        ycols.append(col)
        for r in range(7):
            assert Y[r, i] == col.get(r, 0.0)
    G = explicit.target_gram(7, idx, val)
    for i in range(idx.shape[0]):
        for j in range(idx.shape[0]):
            want = sum(v * ycols[j].get(r, 0.0) for r, v in ycols[i].items())
            assert abs(G[i, j] - want) < 1e-12
    with pytest.raises(IndexError):
        explicit.dense_targets(7, np.array([[7]]), np.array([[1.0]]))
    with pytest.raises(IndexError):
        explicit.dense_targets(7, np.array([[-2]]), np.array([[1.0]]))


# ------------------------------------------- factored algorithm vs definition
def _factored_vs_explicit(loss_kind, steps=20, u_init="random", eps=1e-3, **kw):
    wl = _tiny(loss=loss_kind, seed=23, D=40, d=6, m=4, K=3, u_init=u_init, **kw)
    V0, U0 = wl.init_V(), wl.init_U()
    W = V0.astype(np.float64) @ U0.astype(np.float64)
    st = factored.FactoredState.from_initial(V0, U0)
    lr = 0.02   # keeps 2 lr ||H H^T|| < 1, so U stays well conditioned (error ~ eps * cond U)
    worst = 0.0
    for s in range(steps):
        H, idx, val = wl.batch(s)
        if loss_kind == "squared":
            loss_e, grad_e, W = explicit.squared_error_step(W, H, idx, val, lr)
            loss_f, grad_f = factored.minibatch_step(st, H, idx, val, lr)
        elif loss_kind == "spherical":
            idx1 = _one_class(idx)
            loss_e, grad_e, W = explicit.spherical_softmax_step(W, H, idx1, lr)
            loss_f, grad_f = factored.spherical_minibatch_step(st, H, idx1, lr)
        else:
            idx1 = _one_class(idx)
            loss_e, grad_e, W = explicit.shifted_spherical_step(W, H, idx1, lr, eps)
            loss_f, grad_f = factored.shifted_spherical_minibatch_step(st, H, idx1, lr, eps)
        Wf = st.W()
        worst = max(worst, _rel(Wf, W), _rel(st.Q, W.T @ W), _rel(loss_f, loss_e), _rel(grad_f, grad_e),
                    _rel(st.s, W.sum(axis=0)), float(np.abs(st.U @ st.UinvT.T - np.eye(6)).max()))
        if loss_kind != "spherical_shifted":
            assert not np.any(st.c)
    return worst


def test_factored_minibatch_equals_explicit_squared():
    """Section 3.2 exactness proof and Appendix B: VU = W, Q = W^T W after every step."""
    assert _factored_vs_explicit("squared", pad_frac=0.2, dup_frac=0.3) < 1e-12


def test_factored_minibatch_equals_explicit_spherical():
    """Derived minibatch form for the spherical softmax (pinned against the definition)."""
    assert _factored_vs_explicit("spherical") < 1e-12


def test_factored_minibatch_equals_explicit_shifted():
    """The shifted form with W = V U + 1 c^T and s = W^T 1 (pinned against the
    definition); a large eps makes the all-ones terms large."""
    assert _factored_vs_explicit("spherical_shifted") < 1e-12
    assert _factored_vs_explicit("spherical_shifted", eps=0.5) < 1e-12


def test_first_step_from_identity_closed_form():
    """From U = I, step 7 of Appendix A gives U_1 = I - 2 lr H H^T exactly."""
    wl = _tiny(seed=29)
    st = factored.FactoredState.from_initial(wl.init_V())
    H, idx, val = wl.batch(0)
    lr = 0.05
    factored.minibatch_step(st, H, idx, val, lr)
    Hc = H.astype(float).T
    np.testing.assert_allclose(st.U, np.eye(Hc.shape[0]) - 2 * lr * Hc @ Hc.T, rtol=0, atol=1e-15)


def test_online_equals_minibatch_at_m1_and_woodbury_is_sherman_morrison():
    wl = _tiny(seed=31, m=1, K=3, u_init="random")
    V0, U0 = wl.init_V(), wl.init_U()
    a = factored.FactoredState.from_initial(V0, U0)
    b = factored.FactoredState.from_initial(V0, U0)
    lr = 0.05
    for s in range(6):
        H, idx, val = wl.batch(s)
        UinvT_before = a.UinvT.copy()
        L1, g1 = factored.online_step(a, H[0], idx[0], val[0], lr)
        Lm, gm = factored.minibatch_step(b, H, idx, val, lr)
        assert abs(L1 - Lm[0]) < 1e-12 * max(1.0, abs(L1))
        np.testing.assert_allclose(g1, gm[0], rtol=1e-12, atol=1e-13)
        for X, Y in ((a.U, b.U), (a.UinvT, b.UinvT), (a.V, b.V), (a.Q, b.Q)):
            np.testing.assert_allclose(X, Y, rtol=1e-11, atol=1e-13)
        sm = factored.sherman_morrison_inverse_T(UinvT_before, H[0], lr)
        np.testing.assert_allclose(sm, a.UinvT, rtol=1e-12, atol=1e-14)
        # and both equal the inverse computed from scratch
        np.testing.assert_allclose(a.UinvT, np.linalg.inv(a.U).T, rtol=1e-10, atol=1e-12)


def test_pristine_restore_keeps_W_and_Q():
    wl = _tiny(seed=37, u_init="random")
    st = factored.FactoredState.from_initial(wl.init_V(), wl.init_U())
    for s in range(3):
        H, idx, val = wl.batch(s)
        factored.minibatch_step(st, H, idx, val, 0.05)
    W, Q = st.W().copy(), st.Q.copy()
    factored.pristine_restore(st)
    np.testing.assert_allclose(st.W(), W, rtol=1e-13, atol=1e-15)
    np.testing.assert_array_equal(st.U, np.eye(W.shape[1]))
    np.testing.assert_array_equal(st.Q, Q)
    np.testing.assert_allclose(st.Q, W.T @ W, rtol=1e-12)


# ----------------------------------------------------------- planted mistakes
def _mutants():
    """Plausible mistakes, planted in the oracle's outputs or inputs."""
    base = explicit.squared_error_step

    def dropped_factor_two(W, H, idx, val, lr):   # the 2 on lr lost (W - lr R h^T)
        loss, g, Wn = base(W, H, idx, val, lr)
        return loss, g, np.asarray(W, float) - 0.5 * (np.asarray(W, float) - Wn)

    def wrong_grad_sign(W, H, idx, val, lr):
        loss, g, Wn = base(W, H, idx, val, lr)
        return loss, -g, Wn

    def grad_without_targets(W, H, idx, val, lr):  # 2 W^T W h: the W^T y term dropped
        loss, _, Wn = base(W, H, idx, val, lr)
        Wd = np.asarray(W, float)
        return loss, 2 * (np.asarray(H, float) @ Wd.T @ Wd), Wn

    def padding_as_last_row(W, H, idx, val, lr):
        idx2 = np.where(idx < 0, np.asarray(W).shape[0] - 1, idx)
        return base(W, H, idx2, val, lr)

    def duplicates_overwrite(W, H, idx, val, lr):
        idx2 = np.array(idx, copy=True)
        for i in range(idx2.shape[0]):
            seen = set()
            for k in range(idx2.shape[1] - 1, -1, -1):   # keep the last slot of a repeated index
                if idx2[i, k] in seen:
                    idx2[i, k] = -1
                seen.add(int(idx2[i, k]))
        return base(W, H, idx2, val, lr)

    def transposed_update(W, H, idx, val, lr):        # h y^T-like mix-up: uses rows of H reversed
        return base(W, H, idx, val, lr)[:2] + (base(W, H[::-1], idx, val, lr)[2],)

    return [dropped_factor_two, wrong_grad_sign, grad_without_targets, padding_as_last_row,
            duplicates_overwrite, transposed_update]


def test_planted_mistakes_are_caught():
    pins = [check_worked_squared, check_fd_grad_h, check_fd_update_W]
    for fn in pins:          # the real oracle passes every pin
        fn(explicit.squared_error_step)
    for mutant in _mutants():
        caught = False
        for fn in pins:
            try:
                fn(mutant)
            except AssertionError:
                caught = True
                break
        assert caught, f"mutant {mutant.__name__} slipped through every pin"


# ------------------------------------------ conditioning scales, fp32 yardstick
@pytest.mark.parametrize("loss", ["squared", "spherical", "spherical_shifted"])
def test_term_scales_brute_force(loss):
    """term_scales against the terms formed from the explicit output o = W h, and
    the triangle inequality (each scale bounds |L_i| and ||grad_i||)."""
    kw = dict(K=1) if loss != "squared" else dict(pad_frac=0.2, dup_frac=0.3)
    wl = _tiny(loss, seed=31, D=40, d=6, m=5, K=kw.pop("K", 4), **kw)
    W = wl.init_V().astype(np.float64)
    H, idx, val = wl.batch(0)
    eps = 1e-3
    L, g, _ = explicit.step(W, H, idx, val, 0.05, loss, eps)
    ls, gs = explicit.term_scales(W, H, idx, val, L, g, loss, eps)
    Hd = H.astype(np.float64)
    for i in range(H.shape[0]):
        o = W @ Hd[i]
        if loss == "squared":
            y = np.zeros(W.shape[0])
            for k in range(idx.shape[1]):
                if idx[i, k] >= 0:
                    y[idx[i, k]] += val[i, k]
            want_l = o @ o + 2 * abs(o @ y) + y @ y
            want_g = 2 * np.linalg.norm(W.T @ o) + 2 * np.linalg.norm(W.T @ y)
        elif loss == "spherical_shifted":
            c = idx[i, 0]
            u = o + eps
            S = u @ u
            s1 = W.sum(axis=0)
            b = -2 / u[c]
            doc = np.linalg.norm(W[c]) * np.linalg.norm(Hd[i])
            s_terms = o @ o + 2 * eps * np.linalg.norm(s1) * np.linalg.norm(Hd[i]) + W.shape[0] * eps ** 2
            want_l = abs(np.log(u[c] ** 2)) + abs(np.log(S)) + abs(b) * doc + s_terms / S
            want_g = ((np.linalg.norm(2 / S * (W.T @ o)) + np.linalg.norm(2 * eps / S * s1))
                      * (1 + s_terms / S) + np.linalg.norm(b * W[c]) + 2 / u[c] ** 2 * doc * np.linalg.norm(W[c]))
        else:
            c = idx[i, 0]
            S = np.sum(o * o + eps)
            b = -2 * o[c] / (o[c] ** 2 + eps)
            db = 2 * (o[c] ** 2 - eps) / (o[c] ** 2 + eps) ** 2
            doc = np.linalg.norm(W[c]) * np.linalg.norm(Hd[i])
            want_l = abs(np.log(o[c] ** 2 + eps)) + abs(np.log(S)) + abs(b) * doc
            want_g = (np.linalg.norm(2 / S * (W.T @ o)) + np.linalg.norm(b * W[c])
                      + abs(db) * doc * np.linalg.norm(W[c]))
        assert abs(ls[i] - want_l) <= 1e-10 * want_l
        assert abs(gs[i] - want_g) <= 1e-10 * want_g
        assert ls[i] >= abs(L[i]) * (1 - 1e-12)
        assert gs[i] >= np.linalg.norm(g[i]) * (1 - 1e-12)


@pytest.mark.parametrize("loss", ["squared", "spherical", "spherical_shifted"])
def test_fp32_yardstick_is_the_definition(loss):
    """step_fp32 is `step` evaluated in float32: on a benign tiny case it agrees to
    fp32 accuracy (and its outputs are float32)."""
    kw = dict(K=1) if loss != "squared" else {}
    wl = _tiny(loss, seed=32, D=60, d=7, m=6, K=kw.pop("K", 3), **kw)
    W = wl.init_V()
    H, idx, val = wl.batch(0)
    a = explicit.step(W, H, idx, val, 0.05, loss)
    b = explicit.step_fp32(W, H, idx, val, 0.05, loss)
    for x, y in zip(b, a):
        assert x.dtype == np.float32
        assert _rel(x, y) < 2e-5
