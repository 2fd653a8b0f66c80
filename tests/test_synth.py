"""The seeded input generators: deterministic, row-prefix consistent, and
shaped like the workload recipes."""

import numpy as np

import synth


def test_deterministic_and_prefix_consistent():
    cfg = synth.get_config("mnist", n=70000)
    a = synth.features(cfg, seed=0, n=70000)
    b = synth.features(cfg, seed=0, n=1000)
    np.testing.assert_array_equal(a[:1000], b)
    c = synth.features(cfg, seed=1, n=1000)
    assert not np.array_equal(b, c)


def test_laws():
    for name in ("tiny", "mnist", "cifar", "timit", "imagenet"):
        cfg = synth.get_config(name)
        x = synth.features(cfg, 0, n=2000)
        assert x.dtype == np.float32 and x.shape == (2000, cfg.d)
        if name == "mnist":
            assert abs((x == 0).mean() - 0.8) < 0.01 and x.max() <= 1
        if name == "imagenet":
            assert abs((x == 0).mean() - 0.5) < 0.01 and x.min() >= 0
        if name == "cifar":
            assert 0 <= x.min() and x.max() < 1


def test_labels_and_batches():
    cfg = synth.get_config("tiny")
    w = synth.make_workload(cfg, 0)
    assert w.labels.min() >= 0 and w.labels.max() < cfg.l
    y = w.y(np.arange(10))
    np.testing.assert_array_equal(y.sum(1), 1.0)
    bs = synth.epoch_batches(cfg.n, 256, 0)
    assert sum(len(b) for b in bs) == cfg.n and len(bs[-1]) == cfg.n - 256 * 7
    np.testing.assert_array_equal(np.sort(np.concatenate(bs)), np.arange(cfg.n))
    assert len(np.unique(w.r)) == cfg.s
