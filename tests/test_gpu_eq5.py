"""Eq.5 (threshold +inf) conv at batch sizes that take the position-major task
form: 16-row tiles of 16 images at one output position, each task running
only the K-steps that touch the image at its position.

The reference for the last step is the oracle's conv at T = 1 on the map
[tp <= T-1] (Eq.1 at the last step: those inputs, and only those, have spiked
by then); the oracle's own Eq.5 firing then gives spikes, first-spike times and
potentials.  Every earlier step must hold zero potential and no spike."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
import synth
from parity import assert_close, assert_equal

spk = pytest.importorskip("paper_1903_02440_amd")

pytestmark = pytest.mark.gpu

INF_PM_IMG = 256  # images per position-major task
INF_NW = 4        # 16-feature tiles per task


def ksteps_valid(Cin, H, W, K, pad, stride):
    """(valid K-steps summed over output positions, positions x K-steps): a
    restatement of the host's choice.  Taps are ordered (ky, kx, channel),
    channels rounded up to CP; a K-step covers 32 taps."""
    CP = 4 if Cin <= 4 else -(-Cin // 8) * 8
    Ho, Wo = (H + 2 * pad - K) // stride + 1, (W + 2 * pad - K) // stride + 1
    ksteps = -(-K * K * CP // 32)
    valid = 0
    for y in range(Ho):
        for x in range(Wo):
            for ks in range(ksteps):
                cells = {ks // (CP // 32)} if CP % 32 == 0 else set(range(ks * 32 // CP, min((ks * 32 + 31) // CP, K * K - 1) + 1))
                valid += any(0 <= y * stride + c // K - pad < H and 0 <= x * stride + c % K - pad < W
                             for c in cells if c < K * K)
    return valid, Ho * Wo * ksteps, Ho * Wo


def takes_position_major(B, Cin, H, W, Cout, K, pad, stride):
    valid, total, howo = ksteps_valid(Cin, H, W, K, pad, stride)
    n_ng = -(-(-(-Cout // 16)) // INF_NW)
    return howo <= 64 and valid * 100 <= total * 85 and n_ng * howo * -(-B // INF_PM_IMG) >= 128


EQ5_CASES = [
    # name, B, T, Cin, H, W, Cout, K, pad, stride, p_silent
    ("S3-shape", 300, 15, 250, 4, 4, 200, 5, 2, 1, 0.7),       # second image block partial
    ("cp40", 700, 6, 40, 5, 5, 72, 5, 2, 1, 0.5),              # K-steps straddle taps
    ("stride2", 600, 10, 64, 7, 7, 144, 5, 2, 2, 0.6),
]


def test_cases_take_the_position_major_form():
    for name, B, T, Cin, H, W, Cout, K, pad, st, ps in EQ5_CASES:
        assert takes_position_major(B, Cin, H, W, Cout, K, pad, st), name
    # the S3 shape of the 1000-image workload does too; a 5-image batch does not
    assert takes_position_major(1000, 250, 4, 4, 200, 5, 2, 1)
    assert not takes_position_major(5, 250, 4, 4, 200, 5, 2, 1)


@pytest.mark.parametrize("case", EQ5_CASES, ids=[c[0] for c in EQ5_CASES])
@pytest.mark.parametrize("kind", ["normal", "dyadic"])
def test_eq5_position_major_parity(case, kind, near_log):
    name, B, T, Cin, H, W, Cout, K, pad, st, ps = case
    g = synth.rng(700 + len(name), 1)
    tf_in = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, ps)
    if kind == "dyadic":
        Wt = synth.dyadic_weights(g, (Cout, Cin, K, K), Cin * K * K)
    else:
        Wt = synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05)
    x = torch.from_numpy(tf_in).to("cuda")
    w = torch.from_numpy(Wt).to("cuda")
    if st == 1:
        P, S, tf, vf = spk.spk_conv_fire_first_spike(x, T, w, pad, math.inf)
    else:
        P, S, tf, vf = spk.spk_conv_fire_first_spike_strided(x, T, w, st, pad, math.inf)
    torch.cuda.synchronize()
    P, S, tf, vf = (t.cpu().numpy() for t in (P, S, tf, vf))

    last = orc.conv_times((tf_in > T - 1).astype(np.uint8), 1, Wt, pad, st)[:, 0]  # P[T-1]
    ref = np.zeros((B, T) + last.shape[1:], np.float32)
    ref[:, T - 1] = last
    Po, So, to, vo = orc.fire(ref, math.inf)
    assert not P[:, :T - 1].any() and not S[:, :T - 1].any(), "steps before the last"
    if kind == "dyadic":
        assert_equal(P[:, T - 1], Po[:, T - 1], "P[T-1]")
    else:
        assert_close(P[:, T - 1], Po[:, T - 1], what="P[T-1]")
    # Eq.5 spikes where P[T-1] > 0; a potential within rounding of 0 could go either way
    near = np.abs(Po[:, T - 1]) <= 1e-5 * np.abs(Wt).max() * Cin * K * K
    assert_equal(S[:, T - 1], So[:, T - 1], "spikes", mask=near)
    assert_equal(tf, to, "t_first", mask=near)
    assert_close(vf, vo, what="v_first")
    near_log(f"eq5 position-major {name}/{kind}", int(near.sum()), near.size)
