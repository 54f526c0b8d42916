"""GPU parity of the Appendix C singular-value stabilisation (lst_stabilize)
against oracle.stabilize, through the C ABI.

The oracle takes the appendix's steps in fp64 from the same fp32 initial state
(V0, U0 and the U^{-T} the library computes at creation, inv(U0)^T); the power
iterations start from the same vector of ones (the library applies 2^7 power
iterations as 7 squarings, equal in exact arithmetic).  Compared: the number
of corrections at each end, the singular value estimates, the final U and V,
W = V U (which must not change), and U^{-T} after a reinversion.
"""
import numpy as np
import pytest

from oracle import factored, stabilize
from synth import Workload, WorkloadConfig

from parity_util import rel

pytestmark = pytest.mark.gpu


def _setup(D, d, sigmas, seed):
    import torch

    import paper_1412_7091_amd as lst

    cfg = WorkloadConfig(name="stab", D=D, d=d, m=8, K=2, u_init="spectrum", u_sigma=sigmas,
                         entropy=seed)
    wl = Workload(cfg)
    V0, U0 = wl.init_V(), wl.init_U()
    dev = torch.device("cuda:0")
    layer = lst.FactoredOutputLayer(torch.from_numpy(V0).to(dev), torch.from_numpy(U0).to(dev),
                                    m_max=8, K_max=2)
    return layer, V0, U0


def _run_both(layer, V0, U0, d, lo, hi, max_fixes):
    rep = layer.stabilize(sigma_low=lo, sigma_high=hi, squarings=7, max_fixes=max_fixes,
                          reinvert=1)
    assert layer.sync() == 0
    st = factored.FactoredState.from_initial(V0, U0)
    rounds = stabilize.stabilize_power(st, lo, hi, 2 ** 7, max_fixes, np.ones(d), reinvert_mode=1)
    return rep, st, rounds


def _tol(sigma):
    """fp32 bound for one correction of sigma: its intermediate terms are
    max(sigma, 1/sigma) times the size of the result (U^T u = sigma v is scaled
    by alpha = (1 - sigma)/sigma; V u u^T by beta = sigma - 1), so the result
    carries about 6e-8 * max(sigma, 1/sigma) relative error; 30x margin."""
    return 30 * 6e-8 * max(sigma, 1.0 / sigma) + 2e-6
@pytest.mark.parametrize("d", [40, 37])
def test_stabilize_low_end_matches_oracle(gpu_lib, d):
    layer, V0, U0 = _setup(3000, d, (3e-3, 5e-3), 61 + d)
    W0 = layer.materialize_W().cpu().numpy().astype(np.float64)
    rep, st, rounds = _run_both(layer, V0, U0, d, 1e-2, 100.0, 3)
    assert [r[2] for r in rounds] == [True, True, False, False]
    assert (rep.fixes_low, rep.fixes_high) == (2, 0)
    assert abs(rep.sigma_min - rounds[2][1]) < 1e-4 * rounds[2][1]
    assert abs(rep.sigma_max - rounds[3][1]) < 1e-4 * rounds[3][1]
    Q, U, Uit = (x.cpu().numpy().astype(np.float64) for x in layer.get_state())
    V = layer.get_V().cpu().numpy().astype(np.float64)
    assert rel(U, st.U) < _tol(3e-3)
    assert rel(V, st.V) < _tol(3e-3)
    assert rel(layer.materialize_W().cpu().numpy(), W0) < _tol(3e-3)   # W = V U unchanged
    assert rel(Uit, np.linalg.inv(U).T) < 1e-5                      # refined after each fix
    s = np.linalg.svd(U, compute_uv=False)
    assert s.min() >= 1e-2 and s.max() <= 100.0
    layer.close()


@pytest.mark.parametrize("d", [40, 37])
def test_stabilize_high_end_matches_oracle(gpu_lib, d):
    layer, V0, U0 = _setup(3000, d, (300.0, 150.0), 71 + d)
    W0 = layer.materialize_W().cpu().numpy().astype(np.float64)
    rep, st, rounds = _run_both(layer, V0, U0, d, 1e-3, 100.0, 3)
    assert [r[2] for r in rounds] == [False, True, True, False]
    assert (rep.fixes_low, rep.fixes_high) == (0, 2)
    assert abs(rep.sigma_min - rounds[0][1]) < 1e-4 * rounds[0][1]
    assert abs(rep.sigma_max - rounds[3][1]) < 1e-4 * rounds[3][1]
    Q, U, Uit = (x.cpu().numpy().astype(np.float64) for x in layer.get_state())
    V = layer.get_V().cpu().numpy().astype(np.float64)
    assert rel(U, st.U) < _tol(300.0)
    assert rel(V, st.V) < _tol(300.0)
    assert rel(layer.materialize_W().cpu().numpy(), W0) < _tol(300.0)
    assert rel(Uit, np.linalg.inv(U).T) < 1e-5
    # nothing left to correct: the state does not change (no refinement either)
    before = [x.clone() for x in layer.get_state()]
    rep2 = layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=1,
                           reinvert=1)
    assert (rep2.fixes_low, rep2.fixes_high) == (0, 0)
    import torch
    assert all(torch.equal(b, a) for b, a in zip(before, layer.get_state()))
    layer.close()


def test_stabilize_both_ends_keeps_W(gpu_lib):
    """sigma_min = 2e-4 and sigma_max = 250 at once (cond(U) > 1e6, beyond what
    fp32 resolves): the corrections still bring every singular value into the
    range and leave W unchanged; they need not follow the fp64 oracle."""
    d = 40
    layer, V0, U0 = _setup(3000, d, (2e-4, 1e-3 / 3, 250.0), 61 + d)
    W0 = layer.materialize_W().cpu().numpy().astype(np.float64)
    rep = layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=4,
                          reinvert=1)
    assert rep.fixes_low >= 2 and rep.fixes_high >= 1
    U = layer.get_state()[1].cpu().numpy().astype(np.float64)
    s = np.linalg.svd(U, compute_uv=False)
    assert s.min() >= 1e-3 and s.max() <= 100.0
    assert rel(layer.materialize_W().cpu().numpy(), W0) < _tol(2e-4)
    layer.close()


def test_stabilize_in_range_changes_nothing(gpu_lib):
    import torch

    import paper_1412_7091_amd as lst

    wl = Workload(WorkloadConfig(name="stab0", D=2000, d=32, m=8, K=2, entropy=77))
    V0 = torch.from_numpy(wl.init_V()).cuda()
    layer = lst.FactoredOutputLayer(V0, m_max=8, K_max=2)   # U = I: every singular value is 1
    before = [x.clone() for x in layer.get_state()] + [layer.get_V()]
    rep = layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=2,
                          reinvert=2)   # the refinement of U^{-T} = I is exact
    assert rep.fixes_low == 0 and rep.fixes_high == 0
    assert abs(rep.sigma_min - 1.0) < 1e-6 and abs(rep.sigma_max - 1.0) < 1e-6
    after = list(layer.get_state()) + [layer.get_V()]
    for b, a in zip(before, after):
        assert torch.equal(b, a)
    layer.close()


def test_periodic_stabilize_keeps_c1_literal_exact(gpu_lib):
    """c1 as specified (H ~ N(0,1), lr = 0.01) drives cond(U) past 1e5 within ten
    steps; corrections after every step keep U in [0.1, 10] and the factored
    W equal to the explicitly trained one."""
    import torch

    import paper_1412_7091_amd as lst
    from oracle import explicit
    from synth import get_config

    cfg = get_config("c1")
    wl = Workload(cfg)
    V0 = wl.init_V()
    dev = torch.device("cuda:0")
    layer = lst.FactoredOutputLayer(torch.from_numpy(V0).to(dev), m_max=cfg.m, K_max=cfg.K)
    layer.set_stabilize(1, sigma_low=0.1, sigma_high=10.0, squarings=7, max_fixes=6,
                        reinvert=1)
    W = V0.astype(np.float64)
    worst = 0.0
    for s in range(cfg.steps):
        H, idx, val = wl.batch(s)
        loss, grad = layer.step(*(torch.from_numpy(x).to(dev) for x in (H, idx, val)), cfg.lr)
        assert layer.sync() == 0
        lr_, gr_, W = explicit.squared_error_step(W, H, idx, val, cfg.lr)
        e_l = abs(loss.double().sum().item() - lr_.sum()) / abs(lr_.sum())
        e_g = rel(grad.cpu().numpy(), gr_)
        worst = max(worst, e_l, e_g)
        assert e_l < 1e-4 and e_g < 1e-4, (s, e_l, e_g)
    Wg = layer.materialize_W().cpu().numpy()
    assert rel(Wg, W) < 1e-3
    U = layer.get_state()[1].cpu().numpy().astype(np.float64)
    s = np.linalg.svd(U, compute_uv=False)
    assert s.min() >= 0.1 * 0.99 and s.max() <= 10.0 * 1.01
    layer.close()


def test_stabilize_full_size_c2(gpu_lib):
    """At the benchmark's size (D = 200 000, d = 500): one singular value of U at
    1e-4 is raised to 1 in one pass over V; W is unchanged (checked on sampled
    rows against V0 U0 in fp64) and U lands in range."""
    import torch

    from synth import get_config

    c2 = get_config("c2")
    layer, V0, U0 = _setup(c2.D, c2.d, (1e-4,), 1412)
    rep = layer.stabilize(sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=2,
                          reinvert=1)
    assert rep.fixes_low == 1 and rep.fixes_high == 0
    Q, U, Uit = (x.cpu().numpy().astype(np.float64) for x in layer.get_state())
    s = np.linalg.svd(U, compute_uv=False)
    assert s.min() > 0.99 and s.max() < 1.01
    assert rel(Uit, np.linalg.inv(U).T) < 1e-5
    rows = np.random.default_rng(5).choice(c2.D, 4096, replace=False)
    V = layer.get_V().cpu().numpy()[rows].astype(np.float64)
    W_ref = V0[rows].astype(np.float64) @ U0.astype(np.float64)
    assert rel(V @ U, W_ref) < _tol(1e-4)
    layer.close()
