"""Helpers shared by the GPU parity tests: run the HIP library and the fp64
oracle side by side on the same seeded inputs and measure their distance."""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

from oracle import explicit
from synth import Workload, WorkloadConfig


def rel(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


@dataclasses.dataclass
class StepReport:
    step: int
    loss_rel: float         # |sum L_gpu - sum L_ref| / |sum L_ref|
    loss_max_rel: float     # max_i |L_i,gpu - L_i,ref| / |L_i,ref|
    loss_term_rel: float    # max_i |L_i,gpu - L_i,ref| / (sum of |terms| of L_i)
    grad_rel: float         # ||dG||_F / ||G_ref||_F
    grad_row_rel: float     # max_i ||dg_i|| / ||g_i,ref||
    grad_term_rel: float    # max_i ||dg_i|| / (sum of ||terms|| of g_i)
    rows_equal: bool        # distinct touched rows identical to the oracle's
    W_rel: Optional[float] = None
    yard_grad_rel: Optional[float] = None   # the fp32 evaluation of the definition
    naive_grad_rel: Optional[float] = None  # the library's explicit-W path


def _compare(s, loss_g, grad_g, loss_r, grad_r, W_before, H, idx, val, cfg, rows_ok):
    loss_g = np.asarray(loss_g, dtype=np.float64)
    grad_g = np.asarray(grad_g, dtype=np.float64)
    lsc, gsc = explicit.term_scales(W_before, H, idx, val, loss_r, grad_r, cfg.loss, cfg.sph_eps)
    dl = np.abs(loss_g - loss_r)
    dg = np.linalg.norm(grad_g - grad_r, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        lmax = float(np.max(dl / np.maximum(np.abs(loss_r), 1e-300)))
        lterm = float(np.max(dl / np.maximum(lsc, 1e-300)))
        grow = float(np.max(dg / np.maximum(np.linalg.norm(grad_r, axis=1), 1e-300)))
        gterm = float(np.max(dg / np.maximum(gsc, 1e-300)))
    return StepReport(step=s, loss_rel=abs(float(loss_g.sum() - loss_r.sum()))
                      / max(abs(float(loss_r.sum())), 1e-30),
                      loss_max_rel=lmax, loss_term_rel=lterm, grad_rel=rel(grad_g, grad_r),
                      grad_row_rel=grow, grad_term_rel=gterm, rows_equal=rows_ok)


def run_parity(cfg: WorkloadConfig, steps: int, *, cond_max: float = 0.0, check_rows: bool = True,
               W_every: int = 0, naive: bool = False, V_check_untouched: bool = False,
               yardstick: bool = False, with_naive: bool = False, log_every: int = 0,
               solve: bool = False):
    """Steps the GPU library and the explicit-W oracle from the same initial W.

    yardstick: also step the definition in fp32 on the host (explicit.step_fp32)
    and record its grad distance from the oracle (StepReport.yard_grad_rel).
    with_naive: also step the library's explicit-W (naive) path on the GPU and
    record its grad distance (StepReport.naive_grad_rel).
    solve: step with lst_step_solve (U_new^T Z = H solved from scratch).
    Returns (reports, W_rel_final, extra) where extra holds the final layer object."""
    import torch

    import paper_1412_7091_amd as lst

    wl = Workload(cfg)
    V0 = wl.init_V()
    U0 = wl.init_U()
    dev = torch.device("cuda:0")
    V0_t = torch.from_numpy(V0).to(dev)
    U0_t = None if cfg.u_init == "identity" else torch.from_numpy(U0).to(dev)
    W_ref = V0.astype(np.float64) @ U0.astype(np.float64)
    W0_32 = torch.from_numpy(W_ref.astype(np.float32)).to(dev)
    if naive:
        layer = lst.NaiveOutputLayer(W0_32, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=cfg.m,
                                     K_max=cfg.K)
    else:
        layer = lst.FactoredOutputLayer(V0_t, U0_t, loss=cfg.loss, sph_eps=cfg.sph_eps,
                                        m_max=cfg.m, K_max=cfg.K, cond_max=cond_max)
    side = None
    if with_naive:
        side = lst.NaiveOutputLayer(W0_32, loss=cfg.loss, sph_eps=cfg.sph_eps, m_max=cfg.m,
                                    K_max=cfg.K)
    W_y = W_ref.astype(np.float32) if yardstick else None
    reports: List[StepReport] = []
    V_prev = None
    for s in range(steps):
        H, idx, val = wl.batch(s)
        if V_check_untouched and not naive:
            V_prev = layer.get_V().cpu().numpy()
        H_t = torch.from_numpy(H).to(dev)
        i_t = torch.from_numpy(idx).to(dev)
        v_t = torch.from_numpy(val).to(dev)
        stepper = layer.step_solve if solve else layer.step
        loss_t, grad_t = stepper(H_t, i_t, v_t, cfg.lr)
        code = layer.sync()
        assert code == 0, f"step {s}: device status {code}"
        loss_g = loss_t.cpu().numpy()
        grad_g = grad_t.cpu().numpy()
        W_before = W_ref
        loss_r, grad_r, W_ref = explicit.step(W_ref, H, idx, val, cfg.lr, cfg.loss, cfg.sph_eps)
        rows_ok = True
        if check_rows and not naive:
            rows_ok = bool(np.array_equal(layer.touched_rows(), explicit.touched_rows(idx)))
        rep = _compare(s, loss_g, grad_g, loss_r, grad_r, W_before, H, idx, val, cfg, rows_ok)
        if W_y is not None:
            _, gy, W_y = explicit.step_fp32(W_y, H, idx, val, cfg.lr, cfg.loss, cfg.sph_eps)
            rep.yard_grad_rel = rel(gy, grad_r)
        if side is not None:
            _, gn = side.step(H_t, i_t, v_t, cfg.lr)
            assert side.sync() == 0
            rep.naive_grad_rel = rel(gn.cpu().numpy(), grad_r)
        if W_every and (s + 1) % W_every == 0:
            rep.W_rel = rel(layer.materialize_W().cpu().numpy(), W_ref)
        if V_check_untouched and not naive:
            V_now = layer.get_V().cpu().numpy()
            touched = explicit.touched_rows(idx)
            mask = np.ones(V_now.shape[0], dtype=bool)
            mask[touched] = False
            assert np.array_equal(V_now[mask], V_prev[mask]), f"step {s}: untouched rows of V changed"
        reports.append(rep)
        if log_every and (s % log_every == 0 or s == steps - 1):
            print(f"  step {s}: loss {rep.loss_rel:.1e}/{rep.loss_term_rel:.1e} grad "
                  f"{rep.grad_rel:.1e}/{rep.grad_term_rel:.1e}"
                  + (f" W {rep.W_rel:.1e}" if rep.W_rel is not None else ""), flush=True)
    W_final = layer.materialize_W().cpu().numpy()
    if side is not None:
        side.close()
    return reports, rel(W_final, W_ref), {"layer": layer, "W_ref": W_ref}
