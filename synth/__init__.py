"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds none of the method's arithmetic: it only draws images,
filter banks, weights, labels and first-spike-time maps.  Both the CPU
oracle and the HIP path receive exactly what it returns.

Every generator is driven by ``numpy.random.default_rng([workload_id, stream])``
with stream 0 = images / input waves, 10 + l = layer-l weights, 20 = labels.

Stand-ins (no data set is read or reproduced):
* MNIST-like digits: 28x28 u8 images with a few random thick line strokes
  (value 255) on black -- same size, value range and sparsity as
  handwritten digits, not their content.
* natural images: 1/f-amplitude-spectrum Gaussian noise rescaled to 0..255.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


def rng(workload: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(workload), int(stream)])


# ---------------------------------------------------------------- images
def stroke_images(g: np.random.Generator, B: int, H: int = 28, W: int = 28,
                  n_strokes: int = 3) -> np.ndarray:
    """B images of n_strokes random line segments, widths in {1,2,3}, value 255."""
    yy, xx = np.mgrid[0:H, 0:W].astype(np.float64)
    out = np.zeros((B, H, W), np.uint8)
    for b in range(B):
        m = np.zeros((H, W), bool)
        for _ in range(n_strokes):
            y0, x0, y1, x1 = g.uniform(3, H - 4), g.uniform(3, W - 4), g.uniform(3, H - 4), g.uniform(3, W - 4)
            width = int(g.integers(1, 4))
            dy, dx = y1 - y0, x1 - x0
            L2 = dy * dy + dx * dx
            if L2 == 0:
                s = np.zeros_like(yy)
            else:
                s = np.clip(((yy - y0) * dy + (xx - x0) * dx) / L2, 0.0, 1.0)
            d2 = (yy - (y0 + s * dy)) ** 2 + (xx - (x0 + s * dx)) ** 2
            m |= d2 <= (width / 2.0) ** 2 + 0.25
        out[b][m] = 255
    return out


def pink_noise_images(g: np.random.Generator, B: int, H: int = 160, W: int = 250) -> np.ndarray:
    """B images whose amplitude spectrum falls as 1/f, rescaled to 0..255 u8."""
    fy = np.fft.fftfreq(H)[:, None]
    fx = np.fft.rfftfreq(W)[None, :]
    f = np.sqrt(fy * fy + fx * fx)
    f[0, 0] = 1.0
    out = np.empty((B, H, W), np.uint8)
    for b in range(B):
        spec = np.fft.rfft2(g.standard_normal((H, W))) / f
        spec[0, 0] = 0.0
        im = np.fft.irfft2(spec, s=(H, W))
        lo, hi = im.min(), im.max()
        out[b] = np.round(255.0 * (im - lo) / max(hi - lo, 1e-12)).astype(np.uint8)
    return out


# ---------------------------------------------------------------- filter banks
def _quantize_zero_sum(k: np.ndarray, bits: int = 8) -> np.ndarray:
    """Zero mean, max|k| = 1, then multiples of 2^-bits whose sum is exactly 0
    (the residue goes to the centre tap).  With u8 pixels every product and
    partial sum of the filtering is then exact in float32."""
    k = k - k.mean()
    k = k / np.abs(k).max()
    q = np.round(k * (1 << bits)).astype(np.int64)
    c = k.shape[0] // 2
    q[c, c] -= q.sum()
    return (q.astype(np.float64) / (1 << bits)).astype(np.float32)


def dog_kernel(size: int, s1: float, s2: float) -> np.ndarray:
    r = np.arange(size, dtype=np.float64) - (size - 1) / 2.0
    yy, xx = np.meshgrid(r, r, indexing="ij")
    d2 = yy * yy + xx * xx
    g1 = np.exp(-d2 / (2 * s1 * s1)) / (2 * math.pi * s1 * s1)
    g2 = np.exp(-d2 / (2 * s2 * s2)) / (2 * math.pi * s2 * s2)
    return g1 - g2


def dog_bank(sizes=(3, 7, 13), ratio: float = 2.0) -> np.ndarray:
    """On/off-centre DoG pairs (sigma1 = size/9, sigma2 = ratio*sigma1), each
    quantized and zero-padded (centred) to the largest size.
    Channel order: on3, off3, on7, off7, on13, off13."""
    KF = max(sizes)
    out = []
    for s in sizes:
        on = _quantize_zero_sum(dog_kernel(s, s / 9.0, ratio * s / 9.0))
        for k in (on, -on):
            pad = (KF - s) // 2
            out.append(np.pad(k, pad))
    return np.stack(out).astype(np.float32)


def gabor_bank(size: int = 5, lam: float = 5.0, sigma: float = 2.8, gamma: float = 0.5,
               thetas=(0.0, 45.0, 90.0, 135.0)) -> np.ndarray:
    """Gabor kernels exp(-(x'^2 + gamma^2 y'^2)/(2 sigma^2)) cos(2 pi x'/lam), quantized."""
    r = np.arange(size, dtype=np.float64) - (size - 1) / 2.0
    yy, xx = np.meshgrid(r, r, indexing="ij")
    out = []
    for th in thetas:
        t = math.radians(th)
        xp = xx * math.cos(t) + yy * math.sin(t)
        yp = -xx * math.sin(t) + yy * math.cos(t)
        k = np.exp(-(xp * xp + gamma * gamma * yp * yp) / (2 * sigma * sigma)) * np.cos(2 * math.pi * xp / lam)
        out.append(_quantize_zero_sum(k))
    return np.stack(out).astype(np.float32)


# ---------------------------------------------------------------- weights / labels / times
def normal_weights(g: np.random.Generator, shape, mean: float, std: float,
                   lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    return np.clip(g.normal(mean, std, size=shape), lo, hi).astype(np.float32)


def uniform_weights(g: np.random.Generator, shape, lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    return g.uniform(lo, hi, size=shape).astype(np.float32)


def dyadic_weights(g: np.random.Generator, shape, taps: int) -> np.ndarray:
    """Weights m * 2^-f in [0,1] with f = 24 - ceil(log2(taps + 1)): every
    partial sum of up to `taps` of them is exact in float32."""
    f = 24 - int(math.ceil(math.log2(taps + 1)))
    f = min(f, 20)
    m = g.integers(0, (1 << f) + 1, size=shape)
    return (m.astype(np.float64) / (1 << f)).astype(np.float32)


def loguniform_weights(g: np.random.Generator, shape, decades: float, p_zero: float = 0.0) -> np.ndarray:
    """Weights 10^U(-decades, 0), i.e. spread evenly over `decades` orders of
    magnitude below 1, with a fraction p_zero of exact zeros."""
    w = np.power(10.0, g.uniform(-decades, 0.0, size=shape))
    w[g.random(size=shape) < p_zero] = 0.0
    return w.astype(np.float32)


def labels(g: np.random.Generator, B: int, n_classes: int = 10) -> np.ndarray:
    return g.integers(0, n_classes, size=B).astype(np.int32)


def times_uniform_or_silent(g: np.random.Generator, shape, T: int, p_silent: float) -> np.ndarray:
    """First-spike times: never (T) with probability p_silent, else uniform in 0..T-1."""
    t = g.integers(0, T, size=shape)
    t[g.random(size=shape) < p_silent] = T
    return t.astype(np.uint8)


def times_geometric(g: np.random.Generator, shape, T: int, p: float) -> np.ndarray:
    """First-spike times ~ number of failures before the first success (p);
    values >= T never spike."""
    t = g.geometric(p, size=shape) - 1
    return np.minimum(t, T).astype(np.uint8)


# ---------------------------------------------------------------- workloads
@dataclass
class Conv:
    """A convolutional spiking layer: conv -> fire -> kWTA, then its plasticity rule."""
    cin: int
    cout: int
    K: int
    pad: int
    thr: float
    k: int
    r: int
    learn: str | None = "stdp"  # "stdp", "rstdp" or None
    a_plus: float = 0.004
    a_minus: float = -0.003
    lb: float = 0.0
    ub: float = 1.0
    stabilizer: bool = True
    stride: int = 1


@dataclass
class Pool:
    P: int
    R: int
    D: int = 0


@dataclass
class Workload:
    wid: int
    name: str
    B: int
    T: int
    H: int
    W: int
    stages: list = field(default_factory=list)
    source: str = "image"   # "image": u8 images encoded with `bank`; "wave": first-spike times given
    bank: str | None = None
    cin: int = 1            # input channels of a "wave" source
    n_classes: int = 10


# The five workloads: the paper's tutorial network on MNIST-sized inputs
# (single layer and full 3-layer), a natural-image-sized layer, and two
# stress layers.
def mnist_single(B: int = 1) -> Workload:
    return Workload(1, "mnist-S1", B, 15, 28, 28, [Conv(6, 30, 5, 2, 15.0, 5, 3)], bank="dog")


def mnist_3layer(B: int = 1000) -> Workload:
    return Workload(2, "mnist-3layer", B, 15, 28, 28, [
        Conv(6, 30, 5, 2, 15.0, 5, 3), Pool(2, 2),
        Conv(30, 250, 3, 1, 10.0, 8, 1), Pool(3, 3),
        Conv(250, 200, 5, 2, math.inf, 1, 0, learn="rstdp"),
    ], bank="dog")


def natural_single(B: int = 64) -> Workload:
    return Workload(3, "natural-S2", B, 30, 160, 250, [Pool(7, 6), Conv(4, 20, 17, 0, 36.0, 1, 5)], bank="gabor")


def stress_forward(B: int = 256) -> Workload:
    return Workload(4, "stress-fwd", B, 15, 14, 14, [Conv(30, 250, 3, 1, 10.0, 8, 1, learn=None)],
                    source="wave", cin=30)


def stress_large(B: int = 16) -> Workload:
    return Workload(5, "stress-large", B, 64, 256, 256, [Conv(64, 256, 5, 2, 40.0, 32, 4)], source="wave", cin=64)


WORKLOADS = {1: mnist_single, 2: mnist_3layer, 3: natural_single, 4: stress_forward, 5: stress_large}


def make_inputs(wl: Workload, weights: str = "paper") -> dict:
    """Seeded inputs of a workload: source data, filter bank, labels and one
    weight tensor per conv stage.  weights="dyadic" draws exactly summable
    weights instead (same shapes) for bit-exact checks."""
    out = {}
    g0 = rng(wl.wid, 0)
    if wl.source == "image":
        if wl.bank == "dog":
            out["image"] = stroke_images(g0, wl.B, wl.H, wl.W)
            out["bank"] = dog_bank()
        else:
            out["image"] = pink_noise_images(g0, wl.B, wl.H, wl.W)
            out["bank"] = gabor_bank()
    elif wl.wid == 5:
        out["t_first"] = times_geometric(g0, (wl.B, wl.cin, wl.H, wl.W), wl.T, 0.05)
    else:
        out["t_first"] = times_uniform_or_silent(g0, (wl.B, wl.cin, wl.H, wl.W), wl.T, 0.6)
    out["labels"] = labels(rng(wl.wid, 20), wl.B, wl.n_classes)
    ws = []
    li = 0
    for st in wl.stages:
        if not isinstance(st, Conv):
            continue
        li += 1
        g = rng(wl.wid, 10 + li)
        shape = (st.cout, st.cin, st.K, st.K)
        if weights == "dyadic":
            ws.append(dyadic_weights(g, shape, st.cin * st.K * st.K))
        elif wl.wid == 4:
            ws.append(uniform_weights(g, shape))
        elif wl.wid == 5:
            ws.append(normal_weights(g, shape, 0.5, 0.1))
        else:
            ws.append(normal_weights(g, shape, 0.8, 0.05))
    out["weights"] = ws
    return out
