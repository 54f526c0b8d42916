"""GPU parity of the sparse input layer (section 2.2) against oracle.input_layer,
through the C ABI.  Inputs: the synth generators' (index, value) pairs as the
K-sparse inputs x and their H as dL/dA."""
import numpy as np
import pytest

from oracle import input_layer
from synth import Workload, WorkloadConfig, get_config

from parity_util import rel

pytestmark = pytest.mark.gpu


def _layer(W):
    import torch

    import paper_1412_7091_amd as lst

    return lst.SparseInputLayer(torch.from_numpy(W).cuda())


def _check_steps(cfg, steps, lr):
    import torch

    wl = Workload(cfg)
    W = wl.init_V()
    layer = _layer(W)
    W_ref = W.astype(np.float64)
    for s in range(steps):
        G, idx, val = wl.batch(s)            # G plays dL/dA (m x d)
        i_t, v_t = torch.from_numpy(idx).cuda(), torch.from_numpy(val).cuda()
        A = layer.forward(i_t, v_t).cpu().numpy()
        A_ref = input_layer.forward(W_ref, idx, val)
        # each row is a sum of at most K products: fp32 rounding only
        assert rel(A, A_ref) < 1e-6, (s, rel(A, A_ref))
        W_prev = layer.get_W().cpu().numpy()
        layer.update(i_t, v_t, torch.from_numpy(G).cuda(), lr)
        assert layer.sync() == 0
        W_new = layer.get_W().cpu().numpy()
        W_ref = input_layer.update(W_ref, idx, val, G, lr)
        touched = np.unique(idx[idx >= 0])
        mask = np.ones(W.shape[0], dtype=bool)
        mask[touched] = False
        assert np.array_equal(W_new[mask], W_prev[mask]), "a row no input refers to changed"
        assert rel(W_new[touched], W_ref[touched]) < 1e-6
    layer.close()


@pytest.mark.parametrize("d", [40, 37])
def test_input_layer_small_with_repeats(gpu_lib, d):
    cfg = WorkloadConfig(name="inp", D=300, d=d, m=24, K=6, idx_dist="uniform", distinct=False,
                         val_dist="normal", pad_frac=0.2, dup_frac=0.3, entropy=4000 + d)
    _check_steps(cfg, 4, 0.05)


@pytest.mark.parametrize("d", [300, 37])
def test_input_layer_long_lists(gpu_lib, d):
    """K = 300 > 16: the forward pass splits each list into quarters over four waves."""
    cfg = WorkloadConfig(name="inpl", D=3000, d=d, m=12, K=300, idx_dist="uniform",
                         distinct=False, val_dist="normal", pad_frac=0.1, dup_frac=0.2,
                         entropy=4400 + d)
    _check_steps(cfg, 2, 0.01)


def test_input_layer_zipf_shared_rows(gpu_lib):
    cfg = WorkloadConfig(name="inpz", D=5000, d=64, m=128, K=8, idx_dist="zipf", zipf_s=1.1,
                         distinct=True, val_dist="one", entropy=4100)
    _check_steps(cfg, 3, 0.01)


def test_input_layer_full_size(gpu_lib):
    """D_in = 200 000, d = 500, m = 128 examples with 10 input pairs each."""
    cfg = get_config("c2")
    _check_steps(cfg, 2, 1e-3)


def test_input_layer_max_slots_zipf(gpu_lib):
    """m K = 65 536 slots (the largest call), Zipf 1.1 inputs: rows held by thousands of
    slots next to rows held by one; two calls, so the row table must be left empty."""
    cfg = WorkloadConfig(name="inpmax", D=20000, d=40, m=512, K=128, idx_dist="zipf",
                         zipf_s=1.1, distinct=False, val_dist="normal", entropy=4300)
    _check_steps(cfg, 2, 1e-3)


def test_input_layer_bad_index_leaves_W(gpu_lib):
    import torch

    import paper_1412_7091_amd as lst

    cfg = WorkloadConfig(name="inpb", D=500, d=16, m=8, K=3, entropy=4200)
    wl = Workload(cfg)
    W = wl.init_V()
    layer = _layer(W)
    G, idx, val = wl.batch(0)
    idx[3, 1] = cfg.D                          # out of range
    layer.update(torch.from_numpy(idx).cuda(), torch.from_numpy(val).cuda(),
                 torch.from_numpy(G).cuda(), 0.1)
    assert layer.sync() == lst.LST_EINDEX
    assert np.array_equal(layer.get_W().cpu().numpy(), W)
    # the rejected call still emptied its row table: the next call is exact
    G1, idx1, val1 = wl.batch(1)
    layer.update(torch.from_numpy(idx1).cuda(), torch.from_numpy(val1).cuda(),
                 torch.from_numpy(G1).cuda(), 0.1)
    assert layer.sync() == 0
    W_ref = input_layer.update(W.astype(np.float64), idx1, val1, G1, 0.1)
    assert rel(layer.get_W().cpu().numpy(), W_ref) < 1e-6
    layer.close()
