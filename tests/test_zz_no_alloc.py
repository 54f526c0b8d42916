"""lst_stabilize_noalloc (the static-workspace variant of lst_stabilize, for
callers that cannot allocate) against lst_stabilize, through the C ABI.

Two calls in a row on the same GPU, the second on a smaller state (d = 40,
then d = 24): the static array keeps the first call's contents, which the
second must not read.  Each call runs on a fresh state identical to the one
lst_stabilize corrects; the corrections taken must agree exactly and the
resulting U, U^{-T}, V and Q within fp32 rounding (the same kernels run in
both, so they are expected to agree bit for bit).  A state too large for the
array is refused with LST_ENOSCRATCH before anything runs.
"""
import numpy as np
import pytest

from synth import Workload, WorkloadConfig

from parity_util import rel

pytestmark = pytest.mark.gpu


def _pair(D, d, sigmas, seed):
    import torch

    import paper_1412_7091_amd as lst

    cfg = WorkloadConfig(name="noalloc", D=D, d=d, m=8, K=2, u_init="spectrum", u_sigma=sigmas,
                         entropy=seed)
    wl = Workload(cfg)
    dev = torch.device("cuda:0")
    V0 = torch.from_numpy(wl.init_V()).to(dev)
    U0 = torch.from_numpy(wl.init_U()).to(dev)
    return [lst.FactoredOutputLayer(V0, U0, m_max=8, K_max=2) for _ in range(2)]


def _snapshot(layer):
    return [x.cpu().numpy() for x in layer.get_state()] + [layer.get_V().cpu().numpy()]


@pytest.mark.parametrize("D,d,sigmas,seed", [(3000, 40, (2e-3,), 81), (1500, 24, (300.0,), 82)])
def test_noalloc_matches_stabilize(gpu_lib, D, d, sigmas, seed):
    ref, noa = _pair(D, d, sigmas, seed)
    kw = dict(sigma_low=1e-2, sigma_high=100.0, squarings=7, max_fixes=2, reinvert=1)
    r1 = ref.stabilize(**kw)
    r2 = noa.stabilize_noalloc(**kw)
    assert ref.sync() == 0 and noa.sync() == 0
    assert (r1.fixes_low, r1.fixes_high) == (r2.fixes_low, r2.fixes_high)
    assert r1.fixes_low + r1.fixes_high == 1
    for a, b in ((r1.sigma_min, r2.sigma_min), (r1.sigma_max, r2.sigma_max)):
        assert (np.isnan(a) and np.isnan(b)) or abs(a - b) <= 1e-6 * abs(a)
    same = True
    for x, y, name in zip(_snapshot(ref), _snapshot(noa), ("Q", "U", "UinvT", "V")):
        assert rel(y, x) <= 1e-6, name
        same = same and np.array_equal(x, y)
    print(f"d={d}: corrections {r2.fixes_low}+{r2.fixes_high}, bitwise equal: {same}", flush=True)
    ref.close()
    noa.close()


def test_noalloc_refuses_oversize_state(gpu_lib):
    import torch

    import paper_1412_7091_amd as lst

    dev = torch.device("cuda:0")
    layer = lst.FactoredOutputLayer(torch.zeros((64, 600), device=dev), m_max=1, K_max=1)
    with pytest.raises(lst.LstError) as e:
        layer.stabilize_noalloc()
    assert e.value.code == lst.LST_ENOSCRATCH
    assert layer.sync() == 0
    layer.close()
