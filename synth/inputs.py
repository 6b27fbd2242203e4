"""Seeded synthetic stand-ins for the paper's three datasets plus a stress case.

The paper trains on Fashion-MNIST (latency coded), N-MNIST and SHD (Sec. 3,
App. E). None of those datasets is used here; each configuration below draws
spikes with the shape and coding statistics of one of them, from recipes
written for this project. Every array is a pure function of
(config id, stream, sample index), drawn with NumPy's PCG64:

    stream 0  input spikes (one child stream per batch sample b)
    stream 10+l  weights of LIF layer l (l = 1..L)
    stream 20  readout weights
    stream 30  labels

Spikes are uint8 in time-major layout [T, B, N] (the paper writes B x T x N,
App. E); any nonzero byte is a spike. Weights are float32 [N_in, N_out].
"""
from __future__ import annotations

import json
import math
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

SEED_ROOT = 210508810
_GAINS_PATH = os.path.join(os.path.dirname(__file__), "gains.json")


def rng_for(cfg_id: int, stream: int, *sub: int) -> np.random.Generator:
    """PCG64 generator for (config, stream, sub-keys)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, cfg_id, stream, *sub])))


@dataclass(frozen=True)
class Config:
    """One workload. `sizes` = [N_in, N_1, ..., N_L, C] (L LIF layers, C readout units)."""

    name: str
    cfg_id: int
    T: int
    B: int
    sizes: tuple
    tau_ratio_hidden: float  # dt / tau for LIF layers: alpha = exp(-ratio)
    tau_ratio_out: float  # dt / tau for the readout
    loss_mode: str  # "max" (logits = max over t) or "sum" (logits = sum over t)
    b_th: float  # default backprop band
    b_th_sweep: tuple = ()
    kind: str = "bernoulli"
    rate: float = 0.0  # Bernoulli rate for kind == "bernoulli"
    theta: float = 1.0
    beta: float = 100.0
    description: str = ""
    conv: tuple = ()  # (H, W, C, F) for a convolutional network: sizes = (H W C, H W F, classes)

    @property
    def n_layers(self) -> int:
        return len(self.sizes) - 2

    @property
    def alpha(self) -> np.float32:
        return np.float32(math.exp(-self.tau_ratio_hidden))

    @property
    def alpha_out(self) -> np.float32:
        return np.float32(math.exp(-self.tau_ratio_out))

    def sweep(self) -> tuple:
        return self.b_th_sweep if self.b_th_sweep else (self.b_th,)


CONFIGS = {
    "tiny": Config(
        "tiny", 1, T=20, B=4, sizes=(64, 32, 4), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
        loss_mode="max", b_th=0.2, kind="bernoulli", rate=0.05,
        description="1 LIF layer 64->32, readout 32->4, T=20, B=4, Bernoulli(0.05)"),
    "latency": Config(
        "latency", 2, T=100, B=256, sizes=(784, 200, 10), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
        loss_mode="max", b_th=0.2, kind="latency",
        description="latency code, 784 inputs fire at most once (F-MNIST-like), LIF 784->200, readout 200->10"),
    "event": Config(
        "event", 3, T=300, B=256, sizes=(2312, 200, 10), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
        loss_mode="max", b_th=0.2, b_th_sweep=(0.05, 0.2, 0.5), kind="event",
        description="2x34x34 polarity event stream with clustered bursts (N-MNIST-like), LIF 2312->200, readout 200->10"),
    "audio": Config(
        "audio", 4, T=100, B=256, sizes=(700, 400, 20), tau_ratio_hidden=0.2, tau_ratio_out=0.1,
        loss_mode="sum", b_th=0.2, kind="audio",
        description="700 channels, Poisson spikes under a smooth channel x time envelope (SHD-like), LIF 700->400, readout 400->20"),
    "stress": Config(
        "stress", 5, T=500, B=256, sizes=(1024, 1024, 1024, 1024, 100), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
        loss_mode="max", b_th=0.2, b_th_sweep=(0.02, 0.05, 0.1, 0.2, 0.35, 0.5, 0.8, 1.2), kind="bernoulli", rate=0.02,
        description="3 LIF layers 1024->1024, readout 1024->100, T=500, B=256, Bernoulli(0.02)"),
    "latency_train": Config(
        "latency_train", 6, T=100, B=256, sizes=(784, 200, 200, 10), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
        loss_mode="max", b_th=0.2, kind="classlatency",
        description="class-conditional latency code (F-MNIST-like training task): 28x28 class templates plus "
                    "noise, one spike per input at most; LIF 784->200->200, readout 200->10"),
    "conv": Config(
        "conv", 8, T=100, B=256, sizes=(784, 28 * 28 * 64, 10), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
        loss_mode="max", b_th=0.2, kind="classlatency", conv=(28, 28, 1, 64),
        description="convolutional LIF layer of 64 3x3 filters (padding 1) on the class-conditional latency "
                    "code (28x28x1, F-MNIST-like), 2x2 max pooling, readout 12544->10, T=100, B=256"),
    "deep": Config(
        "deep", 7, T=100, B=256, sizes=(784, 300, 300, 300, 300, 300, 10), tau_ratio_hidden=0.1,
        tau_ratio_out=0.1, loss_mode="max", b_th=0.2, kind="classlatency",
        description="five LIF layers of 300 on the class-conditional latency code (F-MNIST-like): "
                    "784->300->300->300->300->300, readout 300->10, T=100, B=256"),
}


# ---------------------------------------------------------------- input spikes

def _spikes_bernoulli(cfg: Config, b: int) -> np.ndarray:
    r = rng_for(cfg.cfg_id, 0, b)
    return (r.random((cfg.T, cfg.sizes[0])) < cfg.rate).astype(np.uint8)


def _spikes_latency(cfg: Config, b: int) -> np.ndarray:
    """Each input is silent with probability 1/2, else fires once at t ~ U{0..T-1}."""
    r = rng_for(cfg.cfg_id, 0, b)
    n = cfg.sizes[0]
    fires = r.random(n) < 0.5
    when = r.integers(0, cfg.T, size=n)
    x = np.zeros((cfg.T, n), np.uint8)
    idx = np.nonzero(fires)[0]
    x[when[idx], idx] = 1
    return x


EVENT_GRID = 34
EVENT_SIGMA = 2.0
EVENT_BURST_LEN = 20
EVENT_BURSTS_MEAN = 40.0
EVENT_RATE_BG = 0.002
EVENT_RATE_MEAN = 0.010


def event_peak_rate(T: int) -> float:
    """Burst peak rate that makes the expected rate (before clipping) EVENT_RATE_MEAN.

    Expected burst mass = E[K] * p * E[sum_xy gauss] * E[duration]; the grid sum
    is separable in x and y and the centre is uniform on the grid, the onset is
    uniform on {0..T-1} and a burst is cut at T.
    """
    g = EVENT_GRID
    xs = np.arange(g)
    one_d = np.exp(-((xs[None, :] - xs[:, None]) ** 2) / (2 * EVENT_SIGMA ** 2)).sum(1).mean()
    e_space = one_d ** 2
    e_dur = np.minimum(EVENT_BURST_LEN, T - np.arange(T)).mean()
    n_cells = T * 2 * g * g
    return (EVENT_RATE_MEAN - EVENT_RATE_BG) * n_cells / (EVENT_BURSTS_MEAN * e_space * e_dur)


def _spikes_event(cfg: Config, b: int) -> np.ndarray:
    """Polarity x 34 x 34 grid, background rate plus Gaussian bursts; input i = p*1156 + y*34 + x."""
    r = rng_for(cfg.cfg_id, 0, b)
    g, T = EVENT_GRID, cfg.T
    peak = event_peak_rate(T)
    lam = np.full((T, 2, g, g), EVENT_RATE_BG)
    xs = np.arange(g)
    k = r.poisson(EVENT_BURSTS_MEAN)
    cx = r.integers(0, g, size=k)
    cy = r.integers(0, g, size=k)
    pol = r.integers(0, 2, size=k)
    t0 = r.integers(0, T, size=k)
    for n in range(k):
        bump = np.exp(-((xs[:, None] - cy[n]) ** 2 + (xs[None, :] - cx[n]) ** 2) / (2 * EVENT_SIGMA ** 2))
        lam[t0[n]:t0[n] + EVENT_BURST_LEN, pol[n]] += peak * bump
    np.minimum(lam, 1.0, out=lam)
    return (r.random(lam.shape) < lam).reshape(T, 2 * g * g).astype(np.uint8)


AUDIO_MEAN_RATE = 0.02


def _spikes_audio(cfg: Config, b: int) -> np.ndarray:
    """Smooth channel x time envelope (4 Gaussian blobs on a floor), Poisson counts clipped to one spike."""
    r = rng_for(cfg.cfg_id, 0, b)
    n, T = cfg.sizes[0], cfg.T
    c = np.arange(n)[:, None]
    t = np.arange(T)[None, :]
    env = np.full((n, T), 0.2)
    for _ in range(4):
        mu_c = r.uniform(0, n)
        sd_c = r.uniform(20, 80)
        mu_t = r.uniform(0, T)
        sd_t = r.uniform(5, 20)
        a = r.uniform(0.5, 1.0)
        env += a * np.exp(-((c - mu_c) ** 2) / (2 * sd_c ** 2) - ((t - mu_t) ** 2) / (2 * sd_t ** 2))
    lam = env * (AUDIO_MEAN_RATE / env.mean())
    return (r.poisson(lam.T) >= 1).astype(np.uint8)


# Class-conditional latency code for training runs. Each class has a 28x28 template (a few
# Gaussian blobs); a sample adds pixel noise to its class's template and each pixel x above
# LAT_THETA fires once at step floor(LAT_TAU_EFF ln(x / (x - LAT_THETA))) if that is < T
# (brighter pixels fire earlier; tau_eff = 20 steps and theta = 0.2 as in App. E's table).
LAT_TAU_EFF = 20.0
LAT_THETA = 0.2
CLASS_BLOBS = 3
CLASS_NOISE = 0.25
_TEMPLATES = {}


def class_templates(cfg: Config) -> np.ndarray:
    """[C, N_in] float64 intensities in [0, 1] (N_in a square)."""
    if cfg.name not in _TEMPLATES:
        r = rng_for(cfg.cfg_id, 40)
        side = int(round(math.sqrt(cfg.sizes[0])))
        assert side * side == cfg.sizes[0]
        ys, xs = np.mgrid[0:side, 0:side].astype(np.float64)
        out = np.zeros((cfg.sizes[-1], side * side))
        for c in range(cfg.sizes[-1]):
            img = np.zeros((side, side))
            for _ in range(CLASS_BLOBS):
                cy, cx = r.uniform(4, side - 4, 2)
                sd = r.uniform(2.5, 5.0)
                a = r.uniform(0.6, 1.0)
                img += a * np.exp(-((ys - cy) ** 2 + (xs - cx) ** 2) / (2 * sd * sd))
            out[c] = np.clip(img, 0.0, 1.0).ravel()
        _TEMPLATES[cfg.name] = out
    return _TEMPLATES[cfg.name]


def label_of(cfg: Config, sample: int) -> int:
    """Class of one sample of a class-conditional workload (any sample index >= 0)."""
    return int(rng_for(cfg.cfg_id, 30, sample).integers(0, cfg.sizes[-1]))


def _spikes_classlatency(cfg: Config, b: int) -> np.ndarray:
    r = rng_for(cfg.cfg_id, 0, b)
    x = np.clip(class_templates(cfg)[label_of(cfg, b)] + CLASS_NOISE * r.standard_normal(cfg.sizes[0]), 0.0, 1.0)
    out = np.zeros((cfg.T, cfg.sizes[0]), np.uint8)
    idx = np.nonzero(x > LAT_THETA)[0]
    t = np.floor(LAT_TAU_EFF * np.log(x[idx] / (x[idx] - LAT_THETA))).astype(np.int64)
    keep = t < cfg.T
    out[t[keep], idx[keep]] = 1
    return out


_SPIKE_KINDS = {
    "bernoulli": _spikes_bernoulli,
    "latency": _spikes_latency,
    "event": _spikes_event,
    "audio": _spikes_audio,
    "classlatency": _spikes_classlatency,
}


def make_spikes(cfg: Config, batch: Optional[Sequence[int]] = None) -> np.ndarray:
    """Input spikes [T, len(batch), N_in] uint8 for the given batch samples (default: all)."""
    bs = range(cfg.B) if batch is None else batch
    fn = _SPIKE_KINDS[cfg.kind]
    out = np.empty((cfg.T, len(bs), cfg.sizes[0]), np.uint8)
    for k, b in enumerate(bs):
        out[:, k, :] = fn(cfg, int(b))
    return out


# ---------------------------------------------------------------- weights

def load_gains() -> dict:
    if not os.path.exists(_GAINS_PATH):
        return {}
    with open(_GAINS_PATH) as f:
        return json.load(f)


def weight_std(cfg: Config, gains: Optional[dict] = None) -> List[float]:
    """Std of each LIF layer's weights, then the readout's.

    Tiny: N(0, 1/64) for the LIF layer and N(0, 1/32) for the readout.
    Others: sigma_l = kappa_l / sqrt(m_l) with kappa_l = 0.4 sqrt(1 - alpha_l^2),
    m_l = mean spiking inputs per (t, b) row into layer l (frozen in gains.json);
    readout 1/sqrt(N_L).
    """
    L = cfg.n_layers
    if cfg.name == "tiny":
        return [1.0 / 8.0] * L + [1.0 / math.sqrt(cfg.sizes[-2])]
    gains = load_gains() if gains is None else gains
    if cfg.name not in gains:
        raise KeyError(f"weight gains for '{cfg.name}' missing: run synth/calibrate.py")
    return list(gains[cfg.name]["sigma"]) + [1.0 / math.sqrt(cfg.sizes[-2])]


def conv_weight_std(cfg: Config, gains: Optional[dict] = None) -> List[float]:
    """Std of the filters and of the readout of a convolutional workload: filters
    kappa / sqrt(m) with m = mean spiking inputs in a neuron's 3x3xC patch per step (frozen in
    gains.json), readout 1/sqrt((H/2)(W/2)F)."""
    H, W, C, F = cfg.conv
    gains = load_gains() if gains is None else gains
    if cfg.name not in gains:
        raise KeyError(f"weight gains for '{cfg.name}' missing: run synth/calibrate.py")
    return [gains[cfg.name]["sigma"][0], 1.0 / math.sqrt((H // 2) * (W // 2) * F)]


def make_conv_weights(cfg: Config, sigmas: Optional[List[float]] = None):
    """Filters Wc [3, 3, C, F] and readout weights [(H/2)(W/2)F, classes], float32."""
    H, W, C, F = cfg.conv
    sig = conv_weight_std(cfg) if sigmas is None else sigmas
    Wc = (rng_for(cfg.cfg_id, 11).standard_normal((3, 3, C, F)) * sig[0]).astype(np.float32)
    Wo = (rng_for(cfg.cfg_id, 20).standard_normal(((H // 2) * (W // 2) * F, cfg.sizes[-1])) * sig[1]).astype(np.float32)
    return Wc, Wo


@dataclass
class ConvInputs:
    cfg: Config
    X: np.ndarray  # [T, B, H, W, C] uint8
    Wc: np.ndarray
    W_out: np.ndarray
    labels: np.ndarray

    @property
    def alpha(self) -> np.float32:
        return self.cfg.alpha

    @property
    def alpha_out(self) -> np.float32:
        return self.cfg.alpha_out


def make_conv_inputs(cfg: Config, batch: Optional[Sequence[int]] = None, sigmas=None) -> ConvInputs:
    H, W, C, F = cfg.conv
    X = make_spikes(cfg, batch)
    Wc, Wo = make_conv_weights(cfg, sigmas)
    return ConvInputs(cfg=cfg, X=X.reshape(X.shape[0], X.shape[1], H, W, C), Wc=Wc, W_out=Wo,
                      labels=make_labels(cfg, batch))


def make_weights(cfg: Config, sigmas: Optional[List[float]] = None) -> List[np.ndarray]:
    """[W_1, ..., W_L, W_out] float32, W_l of shape [N_{l-1}, N_l]."""
    sig = weight_std(cfg) if sigmas is None else sigmas
    out = []
    for l in range(cfg.n_layers + 1):
        stream = 20 if l == cfg.n_layers else 10 + l + 1
        r = rng_for(cfg.cfg_id, stream)
        out.append((r.standard_normal((cfg.sizes[l], cfg.sizes[l + 1])) * sig[l]).astype(np.float32))
    return out


def make_labels(cfg: Config, batch: Optional[Sequence[int]] = None) -> np.ndarray:
    if cfg.kind == "classlatency":
        bs = range(cfg.B) if batch is None else batch
        return np.array([label_of(cfg, int(b)) for b in bs], np.int32)
    y = rng_for(cfg.cfg_id, 30).integers(0, cfg.sizes[-1], size=cfg.B).astype(np.int32)
    return y if batch is None else y[np.asarray(batch)]


@dataclass
class Inputs:
    cfg: Config
    X: np.ndarray  # [T, B, N_in] uint8
    Ws: List[np.ndarray]  # LIF weights
    W_out: np.ndarray  # readout weights
    labels: np.ndarray  # [B] int32
    batch: Optional[tuple] = None
    alphas: List[np.float32] = field(default_factory=list)

    @property
    def alpha_out(self) -> np.float32:
        return self.cfg.alpha_out


def make_inputs(cfg: Config, batch: Optional[Sequence[int]] = None, sigmas=None) -> Inputs:
    W = make_weights(cfg, sigmas)
    return Inputs(cfg=cfg, X=make_spikes(cfg, batch), Ws=W[:-1], W_out=W[-1],
                  labels=make_labels(cfg, batch), batch=None if batch is None else tuple(batch),
                  alphas=[cfg.alpha] * cfg.n_layers)
