"""The seeded generators: determinism, subsets, and the statistics each recipe promises."""
import numpy as np
import pytest

from synth import CONFIGS, make_inputs
from synth.inputs import make_spikes, event_peak_rate


def test_deterministic_and_subset_equals_slice():
    cfg = CONFIGS["audio"]
    a = make_spikes(cfg, [0, 5, 9])
    b = make_spikes(cfg, [5])
    assert np.array_equal(a[:, 1:2], b)
    assert np.array_equal(a, make_spikes(cfg, [0, 5, 9]))


def test_latency_fires_at_most_once():
    cfg = CONFIGS["latency"]
    x = make_spikes(cfg, range(32))
    per_input = x.sum(axis=0)
    assert per_input.max() == 1
    assert abs(per_input.mean() - 0.5) < 0.02
    assert abs(x.sum(axis=2).mean() - 3.92) < 0.1


@pytest.mark.parametrize("name,rate,tol", [("event", 0.010, 0.0015), ("audio", 0.0198, 0.001),
                                           ("stress", 0.02, 0.0005), ("tiny", 0.05, 0.01)])
def test_mean_rates(name, rate, tol):
    cfg = CONFIGS[name]
    x = make_spikes(cfg, range(min(cfg.B, 24)))
    assert abs(x.mean() - rate) < tol


def test_event_layout_is_polarity_grid():
    cfg = CONFIGS["event"]
    x = make_spikes(cfg, [0])[:, 0].reshape(cfg.T, 2, 34, 34)
    # bursts are spatially clustered: neighbouring pixels co-fire far above chance
    a = x[:, :, :, :-1].astype(float)
    b = x[:, :, :, 1:].astype(float)
    p = x.mean()
    assert (a * b).mean() > 3 * p * p
    assert 0.2 < event_peak_rate(cfg.T) < 0.6


def test_inputs_bundle_shapes():
    for name, cfg in CONFIGS.items():
        inp = make_inputs(cfg, [0, 1])
        assert inp.X.shape == (cfg.T, 2, cfg.sizes[0]) and inp.X.dtype == np.uint8
        assert [W.shape for W in inp.Ws] == [(cfg.sizes[l], cfg.sizes[l + 1]) for l in range(cfg.n_layers)]
        assert inp.W_out.shape == (cfg.sizes[-2], cfg.sizes[-1]) and inp.W_out.dtype == np.float32
        assert inp.labels.shape == (2,) and inp.labels.max() < cfg.sizes[-1]


def test_class_latency_code():
    """Class-conditional latency code: at most one spike per input, brighter template pixels
    fire earlier, labels are a function of the sample index, and classes differ."""
    from synth.inputs import class_templates, label_of, LAT_TAU_EFF, LAT_THETA
    cfg = CONFIGS["latency_train"]
    x = make_spikes(cfg, range(64))
    assert x.sum(axis=0).max() == 1
    y = make_inputs(cfg, range(64)).labels
    assert all(int(y[k]) == label_of(cfg, k) for k in range(64))
    assert np.array_equal(make_inputs(cfg, [70, 3]).labels, [label_of(cfg, 70), label_of(cfg, 3)])
    tm = class_templates(cfg)
    assert tm.shape == (10, 784) and tm.min() >= 0 and tm.max() <= 1
    # a pixel of intensity 1 fires at floor(tau ln(1 / (1 - theta))) without noise
    assert int(np.floor(LAT_TAU_EFF * np.log(1.0 / (1.0 - LAT_THETA)))) == 4
    # mean spike time of bright template pixels is earlier than of dim ones
    t = np.argmax(x, axis=0).astype(float)
    fired = x.sum(axis=0) > 0
    bright = np.array([tm[y[b]] > 0.7 for b in range(64)])
    dim = np.array([tm[y[b]] < 0.1 for b in range(64)])
    assert t[fired & bright].mean() + 5 < t[fired & dim].mean()
    # class templates are distinct
    d = np.abs(tm[:, None] - tm[None]).sum(axis=2)
    assert d[~np.eye(10, dtype=bool)].min() > 10
