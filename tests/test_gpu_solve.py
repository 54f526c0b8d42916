"""GPU parity of the solve-from-scratch step (lst_step_solve): U^{-T} is not
carried; each step forms A = U_new^T, factors it with partial pivoting and
solves A Z = H (section 3.5, last paragraph).  Same bars as the Woodbury step
against the explicit-W oracle, plus agreement with lst_step on the same inputs.
"""
import numpy as np
import pytest
import torch

from parity_util import rel, run_parity
from synth import Workload, WorkloadConfig

pytestmark = pytest.mark.gpu

TOL_STEP = 1e-4
TOL_W = 1e-3


def _cfg(**kw):
    base = dict(name="solve", D=5003, d=70, m=13, K=7, loss="squared", lr=1e-2, steps=30,
                idx_dist="uniform", distinct=False, val_dist="normal", entropy=401)
    base.update(kw)
    return WorkloadConfig(**base)


def _assert(reports, W_rel):
    worst = {k: max(getattr(r, k) for r in reports)
             for k in ("loss_rel", "loss_term_rel", "grad_rel", "grad_term_rel")}
    print(f"steps={len(reports)} " + " ".join(f"{k}={v:.2e}" for k, v in worst.items())
          + f" W rel={W_rel:.2e}", flush=True)
    for r in reports:
        assert r.loss_term_rel <= TOL_STEP, r
        assert r.grad_rel <= TOL_STEP, r
        assert r.grad_term_rel <= TOL_STEP, r
        assert r.rows_equal, r
    assert W_rel <= TOL_W, W_rel


@pytest.mark.parametrize("kw", [
    dict(d=70, m=13, K=7, pad_frac=0.2, dup_frac=0.3),        # rows not 16-byte aligned
    dict(d=37, m=1, K=5),                                      # one example, one ragged panel
    dict(d=130, m=150, K=30, idx_dist="zipf", zipf_s=1.1),     # m > 128, hot rows
    dict(d=96, m=20, K=1, loss="spherical", lr=1e-3, idx_dist="zipf", val_dist="one",
         distinct=True),
])
def test_step_solve_matches_oracle(gpu_lib, kw):
    cfg = _cfg(**kw, entropy=401 + kw["d"] + kw["m"])
    reports, W_rel, _ = run_parity(cfg, 30 if kw["m"] <= 20 else 10, solve=True,
                                   V_check_untouched=True)
    _assert(reports, W_rel)


def test_step_solve_paper_shape(gpu_lib):
    """D = 200000, d = 500, m = 128, K = 10 (the benchmarked shape), 20 steps."""
    cfg = _cfg(D=200000, d=500, m=128, K=10, lr=1e-3, distinct=True, entropy=411)
    reports, W_rel, _ = run_parity(cfg, 20, solve=True)
    _assert(reports, W_rel)


def test_step_solve_agrees_with_woodbury(gpu_lib):
    """The two forms of the step on the same inputs: the same loss, gradient and W
    to fp32 rounding."""
    import paper_1412_7091_amd as lst

    cfg = _cfg(D=4001, d=200, m=64, K=6, lr=5e-3, entropy=412)
    wl = Workload(cfg)
    dev = torch.device("cuda:0")
    V0 = torch.from_numpy(wl.init_V()).to(dev)
    a = lst.FactoredOutputLayer(V0, m_max=cfg.m, K_max=cfg.K)
    b = lst.FactoredOutputLayer(V0, m_max=cfg.m, K_max=cfg.K)
    for s in range(12):
        H, idx, val = (torch.from_numpy(x).to(dev) for x in wl.batch(s))
        la, ga = a.step(H, idx, val, cfg.lr)
        lb, gb = b.step_solve(H, idx, val, cfg.lr)
        assert a.sync() == 0 and b.sync() == 0
        assert rel(lb.cpu().numpy(), la.cpu().numpy()) < 1e-5
        assert rel(gb.cpu().numpy(), ga.cpu().numpy()) < 1e-5
    Wa = a.materialize_W().cpu().numpy()
    Wb = b.materialize_W().cpu().numpy()
    print(f"W rel {rel(Wb, Wa):.2e}", flush=True)
    assert rel(Wb, Wa) < 1e-5
    Qa, Ua, _ = a.get_state()
    Qb, Ub, _ = b.get_state()
    assert rel(Qb.cpu().numpy(), Qa.cpu().numpy()) < 1e-5
    assert rel(Ub.cpu().numpy(), Ua.cpu().numpy()) < 1e-5


def test_step_solve_leaves_uinvt_stale_until_restore(gpu_lib):
    import paper_1412_7091_amd as lst

    cfg = _cfg(D=1500, d=40, m=8, K=4, entropy=413)
    wl = Workload(cfg)
    dev = torch.device("cuda:0")
    layer = lst.FactoredOutputLayer(torch.from_numpy(wl.init_V()).to(dev), m_max=cfg.m,
                                    K_max=cfg.K)
    H, idx, val = (torch.from_numpy(x).to(dev) for x in wl.batch(0))
    layer.step_solve(H, idx, val, cfg.lr)
    assert layer.sync() == 0
    with pytest.raises(lst.LstError) as e:
        layer.step(H, idx, val, cfg.lr)
    assert e.value.code == lst.LST_ESTATE
    with pytest.raises(lst.LstError) as e:
        layer.stabilize()
    assert e.value.code == lst.LST_ESTATE
    W1 = layer.materialize_W().cpu().numpy()
    layer.restore()
    assert rel(layer.materialize_W().cpu().numpy(), W1) < 1e-5
    layer.step(H, idx, val, cfg.lr)
    assert layer.sync() == 0


def test_step_solve_singular(gpu_lib):
    """U = I, lr = 1/8, h = (2, 0, ...): U_new = I - 2 lr h h^T has a zero row and
    column, so the factorisation meets a zero pivot; nothing is updated."""
    import paper_1412_7091_amd as lst

    d, D = 8, 100
    dev = torch.device("cuda:0")
    V0 = torch.from_numpy(Workload(_cfg(D=D, d=d, m=1, K=1)).init_V()).to(dev)
    layer = lst.FactoredOutputLayer(V0, m_max=1, K_max=1)
    before = [x.clone() for x in layer.get_state()[:2]] + [layer.get_V().clone()]
    H = torch.zeros((1, d), dtype=torch.float32, device=dev)
    H[0, 0] = 2.0
    idx = torch.tensor([[3]], dtype=torch.int32, device=dev)
    val = torch.tensor([[1.0]], dtype=torch.float32, device=dev)
    layer.step_solve(H, idx, val, 0.125)
    assert layer.sync() == lst.LST_ESINGULAR
    after = [x.clone() for x in layer.get_state()[:2]] + [layer.get_V().clone()]
    for x, y in zip(before, after):
        assert torch.equal(x, y)


def test_step_solve_refuses_wide_state(gpu_lib):
    import paper_1412_7091_amd as lst

    dev = torch.device("cuda:0")
    V0 = torch.randn((50, 1100), device=dev) * 0.01
    layer = lst.FactoredOutputLayer(V0, m_max=2, K_max=1)
    H = torch.randn((2, 1100), device=dev)
    idx = torch.zeros((2, 1), dtype=torch.int32, device=dev)
    val = torch.ones((2, 1), device=dev)
    with pytest.raises(lst.LstError) as e:
        layer.step_solve(H, idx, val, 1e-3)
    assert e.value.code == lst.LST_EINVAL
