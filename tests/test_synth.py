"""The seeded generators: reproducible, shaped and distributed as configured."""
import numpy as np

from synth import CONFIGS, Workload, WorkloadConfig, bounded_zipf_sampler


def test_reproducible_and_step_dependent():
    wl = Workload(CONFIGS["c1"])
    a, b = wl.batch(3), Workload(CONFIGS["c1"]).batch(3)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    c = wl.batch(4)
    assert not np.array_equal(a[0], c[0]) and not np.array_equal(a[1], c[1])
    np.testing.assert_array_equal(wl.init_V(), Workload(CONFIGS["c1"]).init_V())


def test_shapes_dtypes_and_ranges_c1():
    cfg = CONFIGS["c1"]
    wl = Workload(cfg)
    H, idx, val = wl.batch(0)
    assert H.shape == (16, 32) and H.dtype == np.float32 and H.flags.c_contiguous
    assert idx.shape == (16, 5) and idx.dtype == np.int32
    assert val.shape == (16, 5) and val.dtype == np.float32
    assert idx.min() >= 0 and idx.max() < cfg.D
    for row in idx:
        assert len(set(row.tolist())) == cfg.K           # without replacement
    V = wl.init_V()
    assert V.shape == (2000, 32) and V.dtype == np.float32
    assert np.abs(V).max() <= 0.01 and np.abs(V).max() > 0.009
    np.testing.assert_array_equal(wl.init_U(), np.eye(32, dtype=np.float32))


def test_h_scale_and_value_distributions():
    wl = Workload(CONFIGS["c1s"])
    H, _, _ = wl.batch(0)
    assert 0.1 < H.std() < 0.25                           # N(0,1)/sqrt(32) ~ 0.177
    cfg = WorkloadConfig(name="t", D=1000, d=8, m=64, K=16, idx_dist="zipf", zipf_s=1.1,
                         val_dist="poisson2p1", entropy=3)
    _, idx, val = Workload(cfg).batch(0)
    assert val.min() >= 1 and np.all(val == np.round(val)) and 2.5 < val.mean() < 3.5
    for row in idx:
        assert len(set(row.tolist())) == 16


def test_zipf_head_probability():
    D, s = 200_000, 1.0
    draw = bounded_zipf_sampler(D, s)
    x = draw(np.random.default_rng(0), 400_000)
    assert x.min() >= 0 and x.max() < D
    p0 = 1.0 / np.sum(np.arange(1, D + 1, dtype=float) ** -s)
    assert abs((x == 0).mean() - p0) < 0.003             # P(rank 1) = 1 / H_{D,s} ~ 0.078
    assert (x == 0).mean() > (x == 1).mean() > (x == 9).mean()


def test_padding_and_duplicates_knobs():
    cfg = WorkloadConfig(name="t", D=50, d=4, m=32, K=6, distinct=True, pad_frac=0.2,
                         dup_frac=0.3, entropy=9)
    _, idx, _ = Workload(cfg).batch(0)
    assert (idx == -1).any()
    assert any(len(set(r[r >= 0].tolist())) < (r >= 0).sum() for r in idx)
