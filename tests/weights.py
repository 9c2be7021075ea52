"""Weight tensors for the conv parity cases whose ranges stress the 16-bit
weight terms of the matrix-core contraction.

``learned_weights`` evolves a layer's weights with the oracle's own STDP
(Eq.4, ordered replay) on synthetic winners, so that they take the shape
plasticity gives them -- pushed towards 0 by multiplicative depression and
towards 1 by potentiation -- without any input from the HIP path.
"""
import numpy as np

import oracle as orc
import synth


def learned_weights(W0, updates_per_feature, T, H, W, pad, seed, a_plus=0.004, a_minus=-0.003):
    """W0 after about `updates_per_feature` Eq.4 updates of every feature.

    A fixed 30% of the input neurons are "salient": they spike in the first
    half of the steps with probability 0.9; the others stay silent with
    probability 0.95, else spike in the second half.  Every feature wins at
    its own fixed position and step T//2, once per image, in batches of 64
    images.  Synapses on salient inputs then potentiate towards 1 and the
    others depress towards 0, the bimodal shape plasticity gives weights."""
    Cout, Cin, K, _ = W0.shape
    g = synth.rng(seed, 30)
    Wt = W0.copy()
    B = 64
    Ho, Wo = H + 2 * pad - K + 1, W + 2 * pad - K + 1
    salient = g.random((Cin, H, W)) < 0.3
    fy, fx = g.integers(0, Ho, Cout), g.integers(0, Wo, Cout)
    win = np.stack([np.tile(np.arange(Cout), (B, 1)), np.full((B, Cout), T // 2),
                    np.tile(fy, (B, 1)), np.tile(fx, (B, 1))], axis=2).astype(np.int32)
    nw = np.full(B, Cout, np.int32)
    half = max(1, T // 2)
    for _ in range(-(-updates_per_feature // B)):
        early = g.integers(0, half, (B, Cin, H, W))
        late = g.integers(half, T, (B, Cin, H, W)) if T > half else np.full((B, Cin, H, W), T)
        tf = np.where(salient, np.where(g.random((B, Cin, H, W)) < 0.9, early, T),
                      np.where(g.random((B, Cin, H, W)) < 0.05, late, T)).astype(np.uint8)
        Wt = orc.stdp(Wt, orc.expand_wave(tf, T), pad, win, nw, a_plus, a_minus)
    return Wt


def range_weights(kind, shape, seed, T=15, H=8, W=8, pad=1):
    """Weights of one range case:
    * "loguniform": 10^U(-12, 0) with 10% exact zeros;
    * "tiny-feature": N(0.8, 0.05) except features 0 and Cout-1, whose
      weights lie in [1e-12, 1e-9];
    * "subnormal-feature": N(0.8, 0.05) except feature 1, whose weights are
      float32 subnormals (below 2^-126);
    * "learned": the oracle's STDP applied ~3000 times to every feature
      (depressed weights near 1e-4);
    * "learned-long": ~8000 updates (depressed weights near 1e-10).
    """
    g = synth.rng(seed, 31)
    if kind == "loguniform":
        return synth.loguniform_weights(g, shape, 12.0, 0.1)
    Wt = synth.normal_weights(g, shape, 0.8, 0.05)
    if kind == "tiny-feature":
        Wt[0] = synth.loguniform_weights(g, shape[1:], 3.0) * np.float32(1e-9)
        Wt[-1] = synth.loguniform_weights(g, shape[1:], 3.0) * np.float32(1e-9)
        return Wt
    if kind == "subnormal-feature":
        Wt[1 % shape[0]] = (g.integers(1, 1 << 22, shape[1:]).astype(np.uint32)).view(np.float32)
        return Wt
    if kind in ("learned", "learned-long"):
        n = 3000 if kind == "learned" else 8000
        return learned_weights(Wt, n, T, H, W, pad, seed)
    raise ValueError(kind)


def wide_range_dyadic(g, shape, taps):
    """Exactly summable weights (multiples of 2^-f with f <= 17, every partial
    sum exact in float32) whose range takes the bf16 split: one weight is
    2^(16-f) and one is 2^-f, below 2^-15 of the largest weight's power of
    two.  With at most 17 significant bits each is carried exactly."""
    f = min(24 - int(np.ceil(np.log2(taps + 1))), 17)
    m = g.integers(0, (1 << f) + 1, size=shape)
    Wt = (m.astype(np.float64) / (1 << f)).astype(np.float32)
    flat = Wt.reshape(-1)
    flat[0] = np.float32(2.0 ** (16 - f))
    flat[flat.size // 2] = np.float32(2.0 ** -f)
    return Wt
