"""GPU parity of the single-example step: lst_step with m = 1 (and K <= 256)
runs the two-launch path with the Sherman-Morrison update of U^{-T}
(Algorithm 1, eq. updateU-T).

Two references: the explicit-W oracle, with the bars of the minibatch tests
(per step loss and grad_H within 1e-4, W within 1e-3 after the run, touched
rows bit for bit), and oracle.factored.online_step, which steps the factored
state itself, so that Q, U, U^{-T} and V are compared entry by entry.
"""
import numpy as np
import pytest
import torch

from oracle import explicit, factored
from parity_util import rel, run_parity
from synth import Workload, WorkloadConfig

pytestmark = pytest.mark.gpu

TOL_STEP = 1e-4
TOL_W = 1e-3
TOL_STATE = 1e-4


def _cfg(**kw):
    base = dict(name="online", D=5003, d=37, m=1, K=8, loss="squared", lr=1e-2, steps=40,
                idx_dist="uniform", distinct=False, val_dist="normal", entropy=301)
    base.update(kw)
    return WorkloadConfig(**base)


def _assert(reports, W_rel, tol_step=TOL_STEP, tol_W=TOL_W):
    worst = {k: max(getattr(r, k) for r in reports)
             for k in ("loss_rel", "loss_term_rel", "grad_rel", "grad_term_rel")}
    print(f"steps={len(reports)} " + " ".join(f"{k}={v:.2e}" for k, v in worst.items())
          + f" W rel={W_rel:.2e}", flush=True)
    for r in reports:
        assert r.loss_term_rel <= tol_step, r
        assert r.grad_rel <= tol_step, r
        assert r.grad_term_rel <= tol_step, r
        assert r.rows_equal, r
    assert W_rel <= tol_W, W_rel


def _layer(cfg, **kw):
    import paper_1412_7091_amd as lst

    wl = Workload(cfg)
    dev = torch.device("cuda:0")
    layer = lst.FactoredOutputLayer(torch.from_numpy(wl.init_V()).to(dev), loss=cfg.loss,
                                    sph_eps=cfg.sph_eps, m_max=cfg.m, K_max=cfg.K, **kw)
    return wl, layer


# ------------------------------------------------ against the factored oracle
@pytest.mark.parametrize("d,pad,dup", [(16, 0.0, 0.0), (37, 0.2, 0.3), (130, 0.1, 0.2),
                                       (500, 0.0, 0.0), (1030, 0.1, 0.1), (1088, 0.0, 0.2)])
def test_online_state_matches_factored_oracle(gpu_lib, d, pad, dup):
    """d = 37, 130 and 1030: rows not 16-byte aligned and a ragged last tile; padding
    slots and indices repeated inside the example.  d = 1030 and 1088 exceed 16 tiles
    a side: the partials are finished by a launch of their own."""
    cfg = _cfg(d=d, pad_frac=pad, dup_frac=dup, entropy=301 + d)
    wl, layer = _layer(cfg)
    st = factored.FactoredState.from_initial(wl.init_V())
    dev = torch.device("cuda:0")
    worst_l = worst_g = 0.0
    for s in range(cfg.steps):
        H, idx, val = wl.batch(s)
        loss_t, grad_t = layer.step(*(torch.from_numpy(x).to(dev) for x in (H, idx, val)), cfg.lr)
        assert layer.sync() == 0
        W_before = st.W()
        L, g = factored.online_step(st, H[0], idx[0], val[0], cfg.lr)
        lsc, gsc = explicit.term_scales(W_before, H, idx, val, np.array([L]), g[None, :],
                                        cfg.loss, cfg.sph_eps)
        dl = abs(float(loss_t.cpu().numpy()[0]) - L) / lsc[0]
        dg = np.linalg.norm(grad_t.cpu().numpy()[0].astype(np.float64) - g) / gsc[0]
        worst_l, worst_g = max(worst_l, dl), max(worst_g, dg)
        assert dl <= TOL_STEP and dg <= TOL_STEP, (s, dl, dg)
    Q, U, Uit = (x.cpu().numpy().astype(np.float64) for x in layer.get_state())
    V = layer.get_V().cpu().numpy().astype(np.float64)
    errs = dict(Q=rel(Q, st.Q), U=rel(U, st.U), UinvT=rel(Uit, st.UinvT), V=rel(V, st.V))
    print(f"d={d} loss {worst_l:.1e} grad {worst_g:.1e} "
          + " ".join(f"{k} {v:.1e}" for k, v in errs.items()), flush=True)
    for k, v in errs.items():
        assert v <= TOL_STATE, (k, v)
    assert np.array_equal(Q, Q.T), "Q is not bitwise symmetric"


# ------------------------------------------------ against the explicit oracle
def test_online_paper_shape_explicit(gpu_lib):
    """D = 200000, d = 500, K = 10 (the benchmarked vocabulary and width), one
    example per step."""
    cfg = _cfg(D=200000, d=500, K=10, lr=1e-2, distinct=True, entropy=311)
    reports, W_rel, _ = run_parity(cfg, 40)
    _assert(reports, W_rel)


def test_online_ragged_explicit_untouched_rows(gpu_lib):
    cfg = _cfg(D=2999, d=70, K=12, pad_frac=0.25, dup_frac=0.25, entropy=312)
    reports, W_rel, _ = run_parity(cfg, 60, V_check_untouched=True)
    _assert(reports, W_rel)


def test_online_spherical(gpu_lib):
    cfg = _cfg(D=30011, d=64, K=1, loss="spherical", lr=1e-3, idx_dist="zipf", zipf_s=1.0,
               val_dist="one", distinct=True, entropy=313)
    reports, W_rel, _ = run_parity(cfg, 60, V_check_untouched=True)
    _assert(reports, W_rel)


def test_online_drift_control(gpu_lib):
    """H ~ N(0, 1) at d = 32 and lr = 0.01: 2 lr ||h||^2 is about 0.64, U drifts fast and
    the pristine restore (||U||_F ||U^-T||_F > 3 d) runs during the 80 steps."""
    cfg = _cfg(D=2000, d=32, K=4, lr=1e-2, h_scale=1.0, entropy=314)
    reports, W_rel, extra = run_parity(cfg, 80, cond_max=3.0, W_every=20)
    assert extra["layer"].stats().restores > 0
    for r in reports:
        if r.W_rel is not None:
            assert r.W_rel <= TOL_W, r
    _assert(reports, W_rel)


def test_online_long_target_list_uses_minibatch_path(gpu_lib):
    """K = 300 exceeds the single-example path's 256 slots: the minibatch path runs
    with m = 1, to the same bars."""
    cfg = _cfg(D=20011, d=48, K=300, lr=5e-3, pad_frac=0.1, dup_frac=0.1, entropy=315)
    reports, W_rel, _ = run_parity(cfg, 10)
    _assert(reports, W_rel)


# ---------------------------------------------------------------- invariants
def test_online_determinism_and_stats(gpu_lib):
    cfg = _cfg(D=3000, d=96, K=16, lr=5e-3, idx_dist="zipf", zipf_s=1.1, dup_frac=0.2,
               pad_frac=0.1, entropy=316)
    dev = torch.device("cuda:0")
    runs = []
    for _ in range(2):
        wl, layer = _layer(cfg)
        outs = []
        for s in range(15):
            H, idx, val = (torch.from_numpy(x).to(dev) for x in wl.batch(s))
            loss, grad = layer.step(H, idx, val, cfg.lr)
            outs.append((loss.clone(), grad.clone()))
        assert layer.sync() == 0
        runs.append((layer, outs))
    (a, oa), (b, ob) = runs
    for x, y in zip(a.get_state(), b.get_state()):
        assert torch.equal(x, y)
    assert torch.equal(a.get_V(), b.get_V())
    for (la, ga), (lb, gb) in zip(oa, ob):
        assert torch.equal(la, lb) and torch.equal(ga, gb)
    _, idx, _ = Workload(cfg).batch(14)
    st = a.stats()
    assert st.last_nnz == int((idx >= 0).sum())
    assert st.last_unique == len(explicit.touched_rows(idx))


def test_online_graph_replay_matches_eager(gpu_lib):
    import paper_1412_7091_amd as lst

    for loss in ("squared", "spherical"):
        kw = dict(K=1, val_dist="one", distinct=True, idx_dist="zipf") if loss == "spherical" \
            else dict(K=6)
        cfg = _cfg(D=3000, d=64, loss=loss, lr=5e-3, entropy=317, **kw)
        wl = Workload(cfg)
        dev = torch.device("cuda:0")
        V0 = torch.from_numpy(wl.init_V()).to(dev)
        layers = [lst.FactoredOutputLayer(V0, loss=loss, m_max=1, K_max=cfg.K) for _ in range(2)]
        layers[0].set_graphs(True)
        layers[1].set_graphs(False)
        bufs = [tuple(torch.from_numpy(x).to(dev) for x in wl.batch(s)) for s in range(3)]
        outs = [[], []]
        for s in range(12):
            H, idx, val = bufs[s % 3]
            for li, layer in enumerate(layers):
                loss_t, grad_t = layer.step(H, idx, val, cfg.lr)
                outs[li].append((loss_t.clone(), grad_t.clone()))
            torch.cuda.synchronize()
            _ = (H * 2).sum().item()
        for layer in layers:
            assert layer.sync() == 0
        for (la, ga), (lb, gb) in zip(*outs):
            assert torch.equal(la, lb) and torch.equal(ga, gb)
        for x, y in zip(layers[0].get_state(), layers[1].get_state()):
            assert torch.equal(x, y)
        assert torch.equal(layers[0].get_V(), layers[1].get_V())


# --------------------------------------------------------------------- errors
def test_online_bad_index_leaves_state_unchanged(gpu_lib):
    import paper_1412_7091_amd as lst

    cfg = _cfg(D=500, d=20, K=3, entropy=318)
    wl, layer = _layer(cfg)
    dev = torch.device("cuda:0")
    for s in range(3):
        layer.step(*(torch.from_numpy(x).to(dev) for x in wl.batch(s)), cfg.lr)
    assert layer.sync() == 0
    before = [x.clone() for x in layer.get_state()] + [layer.get_V().clone()]
    H, idx, val = wl.batch(5)
    idx[0, 1] = cfg.D
    layer.step(*(torch.from_numpy(x).to(dev) for x in (H, idx, val)), cfg.lr)
    assert layer.sync() == lst.LST_EINDEX
    after = [x.clone() for x in layer.get_state()] + [layer.get_V().clone()]
    for x, y in zip(before, after):
        assert torch.equal(x, y)
    layer.step(*(torch.from_numpy(x).to(dev) for x in wl.batch(6)), cfg.lr)
    assert layer.sync() == 0


def test_online_spherical_requires_a_class(gpu_lib):
    import paper_1412_7091_amd as lst

    dev = torch.device("cuda:0")
    V0 = torch.from_numpy(Workload(_cfg(D=50, d=8, K=1)).init_V()).to(dev)
    layer = lst.FactoredOutputLayer(V0, loss="spherical", m_max=1, K_max=1)
    before = [x.clone() for x in layer.get_state()] + [layer.get_V().clone()]
    layer.step(torch.randn((1, 8), device=dev), torch.tensor([[-1]], dtype=torch.int32,
                                                             device=dev), None, 0.01)
    assert layer.sync() == lst.LST_EINDEX
    for x, y in zip(before, [x.clone() for x in layer.get_state()] + [layer.get_V().clone()]):
        assert torch.equal(x, y)
