"""The seeded input generator: determinism and the stated recipe (no GPU)."""
import numpy as np

import synth


def test_deterministic_and_seed_sensitive():
    a = synth.gen_weight(256, 256, 42)
    b = synth.gen_weight(256, 256, 42)
    c = synth.gen_weight(256, 256, 43)
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    x1 = synth.gen_act(8, 256, 42)
    x2 = synth.gen_act(16, 256, 42)
    assert x1.dtype == np.float16 and np.array_equal(x1, x2[:8])


def test_weight_recipe():
    W = synth.gen_weight(1024, 1024, 7)
    assert W.dtype == np.float32
    big = np.abs(W) > 0.2          # outliers are ~20x a 0.02-sigma normal
    frac = big.mean()
    assert 0.003 < frac < 0.006
    assert abs(W[~big].std() - 0.02) < 0.001


def test_act_recipe():
    X = synth.gen_act(512, 1024, 3).astype(np.float32)
    ch_std = X.std(axis=0)
    hot = np.flatnonzero(ch_std > 10)
    assert hot.size == synth.N_OUTLIER_CH
    assert np.all(np.abs(ch_std[hot] - 30) < 4)


def test_budget_and_workloads():
    assert synth.budget(1024, 1024, 10) == 6
    assert synth.budget(4096, 4096, 10) == 102
    assert synth.budget(14336, 4096, 20) == 717
    assert synth.budget(28672, 8192, 10) == 1434
    names = [w.name for w in synth.workloads()]
    assert len(names) == len(set(names)) == 16
    for w in synth.workloads():
        assert w.K % 128 == 0 and w.N % 128 == 0


def test_skew_bands():
    N, K = 5120, 5120
    nnzb = synth.budget(N, K, 10)
    des, n_hot = synth.skew_blocks(N, K, nnzb, 9)
    assert des.sum() == nnzb
    rows = des.sum(axis=1)
    top8 = np.sort(rows)[-8:].sum()
    assert top8 >= n_hot == 128
