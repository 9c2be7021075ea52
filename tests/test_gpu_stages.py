"""Stage-isolated parity: every libspyke call against the oracle on the same
seeded inputs, at sizes spanning several tiles with ragged tails, plus the
edge cases of each call.  Runs through the C ABI on the GPU."""
import functools
import math

import numpy as np
import pytest
import torch

import oracle as orc
import synth
import weights
from parity import assert_close, assert_equal, compare_conv_fire

spk = pytest.importorskip("paper_1903_02440_amd")

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    return t.cpu().numpy()


def dev_shifted(a, shift=1):
    """A device copy of `a` that starts `shift` elements into its allocation,
    so that its address is not aligned to the element group the kernels'
    wide loads use."""
    a = np.ascontiguousarray(a)
    flat = torch.empty(a.size + shift, dtype=torch.from_numpy(a[:0].reshape(-1)).dtype, device="cuda")
    view = flat[shift:].view(a.shape)
    view.copy_(torch.from_numpy(a))
    return view


def sync():
    torch.cuda.synchronize()


def wave_of(tf, T):
    """Eq.1 written directly with numpy (input preparation only)."""
    return (np.arange(T, dtype=np.int32)[None, :, None, None, None] >= tf[:, None].astype(np.int32)).astype(np.uint8)


# ---------------------------------------------------------------- conv + fire
def gpu_conv(wave, W, pad, thr):
    out = spk.spk_conv_fire(dev(wave), dev(W), pad, thr)
    sync()
    return tuple(host(x) for x in out)


def test_conv_toy_t1(golden):
    g = golden("t1_conv_fire.txt")
    T = int(g["T"][0])
    wave = g["wave_in"].astype(np.uint8)
    W = g["weight"].astype(np.float32)
    for thr, key in ((1.875, "a"), (2.0, "b"), (3.0, "c")):
        P, S, tf, vf = gpu_conv(wave, W, 0, thr)
        assert_equal(P, g["potentials"].astype(np.float32), "P")
        assert_equal(tf, g["t_first_" + key].astype(np.uint8), "t_first")
    P, S, tf, vf = gpu_conv(wave, W, 0, 1.875)
    assert_equal(S, g["spikes_a"].astype(np.uint8), "spikes")
    assert vf.item() == np.float32(1.875)
    P, S, tf, vf = gpu_conv(wave, W, 0, math.inf)
    assert_equal(P, g["potentials_inf"].astype(np.float32), "P inf")
    assert_equal(S, g["spikes_inf"].astype(np.uint8), "S inf")
    assert tf.item() == 2 and vf.item() == np.float32(2.625)
    P, S, tf, vf = gpu_conv(wave, W, 1, 100.0)
    assert_equal(P[0, :, 0, 0, 0], g["potentials_pad1_00"].astype(np.float32), "P pad")


CONV_CASES = [
    # name, B, T, Cin, H, W, Cout, K, pad, thr, p_silent
    ("mnist-S1", 3, 15, 6, 28, 28, 30, 5, 2, 15.0, 0.5),
    ("mnist-S2", 2, 15, 30, 14, 14, 250, 3, 1, 10.0, 0.6),
    ("mnist-S3-inf", 5, 15, 250, 4, 4, 200, 5, 2, math.inf, 0.7),
    ("natural-S2", 2, 30, 4, 26, 41, 20, 17, 0, 36.0, 0.5),
    ("T64-ragged", 2, 64, 8, 12, 11, 40, 5, 2, 12.0, 0.4),
    ("odd-sizes", 3, 7, 3, 5, 9, 17, 3, 0, 1.0, 0.5),
    ("tiny", 1, 1, 1, 1, 1, 1, 1, 0, 0.5, 0.3),
    ("inf-small", 3, 4, 2, 6, 6, 5, 3, 1, math.inf, 0.5),
    ("K1", 2, 5, 7, 3, 5, 33, 1, 0, 2.0, 0.3),
    # 9, 10, 13 and 14 position tiles per image, enough of them for whole-image
    # tasks (8 feature pairs): the feature halves of the last tile (9, 13) or of
    # the last two tiles (10, 14) go to two waves each
    ("tiles9-split", 57, 9, 12, 12, 12, 256, 3, 1, 4.0, 0.4),
    ("tiles10-split", 52, 9, 12, 12, 13, 256, 3, 1, 4.0, 0.4),
    ("tiles13-split", 40, 15, 16, 14, 14, 256, 3, 1, 6.0, 0.5),
    ("tiles14-split", 37, 15, 16, 16, 14, 256, 3, 1, 6.0, 0.5),
    # Eq.5 on few tasks: the K chunks split over workgroups, two chunks per part
    ("inf-ksplit", 112, 15, 64, 12, 12, 8, 5, 2, math.inf, 0.6),
]


def fin_task_form(B, Cout, Ho, Wo):
    """How the finite-threshold conv call cuts its work (a restatement of the
    host plan): ("image", split) when each task is one whole image, split being
    whether the last tile's feature halves go to two waves; ("chunks", False)
    for chunks of the flattened position space."""
    mt = -(-Ho * Wo // 16)
    n_pairs = -(-(-(-Cout // 16)) // 2)
    ct = 16 if (Ho * Wo) % 4 == 0 else 8
    while ct > 4 and n_pairs * B * mt // ct < 256:
        ct //= 2
    if mt > ct:
        return ("chunks", False)
    return ("image", (mt & 3) in (1, 2) and mt > 8 and ct == 16)


def test_split_cases_take_the_whole_image_split():
    for name in ("tiles9-split", "tiles10-split", "tiles13-split", "tiles14-split"):
        _, B, T, Cin, H, W, Cout, K, pad, thr, ps = next(c for c in CONV_CASES if c[0] == name)
        assert fin_task_form(B, Cout, H + 2 * pad - K + 1, W + 2 * pad - K + 1) == ("image", True), name


@pytest.mark.parametrize("case", CONV_CASES, ids=[c[0] for c in CONV_CASES])
@pytest.mark.parametrize("kind", ["normal", "dyadic"])
def test_conv_fire_parity(case, kind, near_log):
    name, B, T, Cin, H, W, Cout, K, pad, thr, ps = case
    g = synth.rng(100 + len(name), 1)
    tf = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, ps)
    wave = wave_of(tf, T)
    if kind == "dyadic":
        Wt = synth.dyadic_weights(g, (Cout, Cin, K, K), Cin * K * K)
    else:
        Wt = synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05)
    gpu = gpu_conv(wave, Wt, pad, thr)
    ref = orc.conv_fire(wave, Wt, pad, thr)
    near_log(f"conv {name}/{kind}", compare_conv_fire(gpu, ref, thr, exact_potentials=(kind == "dyadic")),
             ref[2].size)
    if kind == "dyadic" and not math.isinf(thr):
        # exact arithmetic leaves nothing near threshold unresolved
        assert_equal(gpu[1], ref[1], "spikes (exact)")


@pytest.mark.parametrize("case", CONV_CASES, ids=[c[0] for c in CONV_CASES])
def test_conv_fire_first_spike_input(case, near_log):
    # the first-spike-map entry on the map of an Eq.1 wave: oracle parity on the wave, and
    # bitwise the same outputs as the wave entry
    name, B, T, Cin, H, W, Cout, K, pad, thr, ps = case
    g = synth.rng(150 + len(name), 1)
    tf = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, ps)
    wave = wave_of(tf, T)
    Wt = synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05)
    got = spk.spk_conv_fire_first_spike(dev(tf), T, dev(Wt), pad, thr)
    via_wave = spk.spk_conv_fire(dev(wave), dev(Wt), pad, thr)
    sync()
    for a, b in zip(got, via_wave):
        assert torch.equal(a, b)
    ref = orc.conv_fire(wave, Wt, pad, thr)
    near_log(f"conv first-spike input {name}", compare_conv_fire(tuple(host(x) for x in got), ref, thr), ref[2].size)


@pytest.mark.parametrize("case", [c for c in CONV_CASES if not math.isinf(c[9])], ids=lambda c: c[0])
@pytest.mark.parametrize("kind", ["normal", "dyadic", "loguniform"])
def test_conv_fire_f32mfma_parity(case, kind, near_log):
    # the dense fp32 form of the contraction: the oracle's potentials within 1e-5 (exactly
    # summable weights: bit-exact), spikes and first-spike times under the parity rules
    name, B, T, Cin, H, W, Cout, K, pad, thr, ps = case
    g = synth.rng(160 + len(name), 1)
    tf = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, ps)
    if kind == "dyadic":
        Wt = synth.dyadic_weights(g, (Cout, Cin, K, K), Cin * K * K)
    elif kind == "loguniform":
        Wt = synth.loguniform_weights(g, (Cout, Cin, K, K), 12.0, 0.1)
        thr = 0.37
    else:
        Wt = synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05)
    got = spk.spk_conv_fire_first_spike_f32mfma(dev(tf), T, dev(Wt), pad, thr)
    sync()
    ref = orc.conv_fire(wave_of(tf, T), Wt, pad, thr)
    near_log(f"conv f32mfma {name}/{kind}",
             compare_conv_fire(tuple(host(x) for x in got), ref, thr, exact_potentials=(kind == "dyadic")),
             ref[2].size)


# Weight ranges that the 16-bit terms of the contraction must carry: the
# layer shapes of the workloads (finite threshold and Eq.5), the natural
# layer whose fragments are read from the workspace, and a ragged small case.
RANGE_SHAPES = [
    # name, B, T, Cin, H, W, Cout, K, pad, thr
    ("S1", 3, 15, 6, 28, 28, 30, 5, 2, 1.37),
    ("S2", 2, 15, 30, 14, 14, 250, 3, 1, 1.43),
    ("S3-inf", 5, 15, 250, 4, 4, 200, 5, 2, math.inf),
    ("natural", 2, 30, 4, 26, 41, 20, 17, 0, 2.71),
    ("ragged", 3, 7, 3, 5, 9, 17, 3, 0, 0.37),
]
# (thresholds away from integers: plasticity leaves weights just below 1, so
# potentials sit near whole numbers)
RANGE_KINDS = ["loguniform", "tiny-feature", "subnormal-feature", "learned", "learned-long"]


@functools.lru_cache(maxsize=None)
def _range_weights(kind, shape_name):
    name, B, T, Cin, H, W, Cout, K, pad, thr = next(c for c in RANGE_SHAPES if c[0] == shape_name)
    return weights.range_weights(kind, (Cout, Cin, K, K), 40 + len(name), T, H, W, pad)


@pytest.mark.parametrize("case", RANGE_SHAPES, ids=[c[0] for c in RANGE_SHAPES])
@pytest.mark.parametrize("kind", RANGE_KINDS)
def test_conv_fire_weight_range(case, kind, near_log):
    # potentials within 1e-5 relative of the oracle's (exact zeros exactly) for
    # weights spread over 12 decades, features far below the layer's largest
    # weight, subnormal weights and weights shaped by plasticity
    name, B, T, Cin, H, W, Cout, K, pad, thr = case
    if kind == "learned-long" and Cin * K * K > 1000:
        pytest.skip("the oracle's plasticity run takes minutes at this size; the smaller layers cover it")
    g = synth.rng(170 + len(name), 1)
    tf = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5)
    wave = wave_of(tf, T)
    Wt = _range_weights(kind, name)
    gpu = gpu_conv(wave, Wt, pad, thr)
    ref = orc.conv_fire(wave, Wt, pad, thr)
    n_near = compare_conv_fire(gpu, ref, thr)
    near_log(f"conv weight-range {name}/{kind}", n_near, ref[2].size)
    assert n_near <= ref[2].size // 100, "the case leaves too many neurons near the threshold to test spikes"


@pytest.mark.parametrize("case", RANGE_SHAPES, ids=[c[0] for c in RANGE_SHAPES])
def test_conv_fire_bf16_split_exact(case):
    # exactly summable weights of at most 17 significant bits whose range takes
    # the bf16 split: bit-exact
    name, B, T, Cin, H, W, Cout, K, pad, thr = case
    g = synth.rng(180 + len(name), 1)
    tf = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5)
    wave = wave_of(tf, T)
    Wt = weights.wide_range_dyadic(g, (Cout, Cin, K, K), Cin * K * K)
    thr = math.inf if math.isinf(thr) else float(np.float32(0.37 * Cin * K * K))
    gpu = gpu_conv(wave, Wt, pad, thr)
    ref = orc.conv_fire(wave, Wt, pad, thr)
    for x, r, what in zip(gpu, ref, ("P", "S", "t_first", "v_first")):
        assert_equal(x, r, what)


def test_conv_fire_deterministic_and_optional_outputs():
    B, T, Cin, H, W, Cout, K, pad = 2, 15, 30, 14, 14, 250, 3, 1
    g = synth.rng(7, 1)
    wave = dev(wave_of(synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5), T))
    Wt = dev(synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05))
    a = spk.spk_conv_fire(wave, Wt, pad, 10.0)
    b = spk.spk_conv_fire(wave, Wt, pad, 10.0)
    _, _, tf, vf = spk.spk_conv_fire(wave, Wt, pad, 10.0, potentials=False, spikes=False)
    sync()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    assert torch.equal(tf, a[2]) and torch.equal(vf, a[3])


def test_conv_fire_unaligned_wave():
    B, T, Cin, H, W, Cout, K, pad = 2, 15, 6, 28, 28, 30, 5, 2
    g = synth.rng(8, 1)
    wave = wave_of(synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5), T)
    Wt = synth.dyadic_weights(g, (Cout, Cin, K, K), Cin * K * K)
    out = spk.spk_conv_fire(dev_shifted(wave), dev(Wt), pad, 15.0)
    sync()
    ref = orc.conv_fire(wave, Wt, pad, 15.0)
    for x, r, name in zip(out, ref, ("P", "S", "t_first", "v_first")):
        assert_equal(host(x), r, name)


# ---------------------------------------------------------------- synaptic events
@pytest.mark.parametrize("case", [(3, 15, 6, 28, 28, 30, 5, 2), (5, 15, 30, 14, 14, 250, 3, 1),
                                  (7, 15, 250, 4, 4, 200, 5, 2), (2, 30, 4, 26, 41, 20, 17, 0),
                                  (3, 7, 3, 5, 9, 17, 3, 1), (1, 4, 2, 3, 3, 1, 3, 0), (13, 9, 5, 7, 7, 11, 3, 2)])
def test_count_events_parity(case):
    # batch * output positions not a multiple of 64 in the last cases (the reduction's tail), padding in most
    B, T, Cin, H, W, Cout, K, pad = case
    g = synth.rng(140 + H + Cin, 0)
    tf = synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.6)
    count = spk.spk_count_events(dev(wave_of(tf, T)), Cout, K, pad)
    sync()
    assert int(count.item()) == orc.count_events(tf, T, Cout, K, pad)


# ---------------------------------------------------------------- pool
# (B, T, C, H, W, P, R, D).  First-spike pooling stages whole planes in LDS
# (blocks of channels) when C*Ho*Wo is a multiple of 4 and a plane holds at
# most 16 KB: the first two (a partial last block), (4x4 window with padding)
# and (odd 5x5 output planes); the 160x250 planes and the rest take the
# direct paths.
POOL_CASES = [(3, 15, 30, 28, 28, 2, 2, 0), (2, 15, 250, 14, 14, 3, 3, 0), (2, 30, 4, 160, 250, 7, 6, 0),
              (2, 7, 3, 9, 10, 3, 2, 1), (1, 5, 2, 5, 5, 5, 1, 2), (2, 3, 1, 1, 1, 1, 1, 0),
              (2, 9, 8, 12, 12, 4, 2, 1), (2, 5, 12, 10, 10, 2, 2, 0),
              # batches of a few hundred images
              (256, 15, 30, 8, 8, 2, 2, 0), (260, 15, 25, 9, 9, 3, 3, 0)]


@pytest.mark.parametrize("case", POOL_CASES)
def test_pool_parity(case):
    B, T, C, H, W, P, R, D = case
    g = synth.rng(200 + H, 0)
    tf = synth.times_uniform_or_silent(g, (B, C, H, W), T, 0.7)
    wave = wave_of(tf, T)
    out, otf = spk.spk_pool(dev(wave), P, R, D, out_t_first=None)
    sync()
    ref = orc.pool(wave, P, R, D)
    assert_equal(host(out), ref, "pooled wave")
    assert_equal(host(otf), orc.first_spike(ref), "pooled t_first")


@pytest.mark.parametrize("case", POOL_CASES)
def test_pool_first_spike_parity(case):
    B, T, C, H, W, P, R, D = case
    g = synth.rng(250 + H, 0)
    tf = synth.times_uniform_or_silent(g, (B, C, H, W), T, 0.7)
    out, otf = spk.spk_pool_first_spike(dev(tf), T, P, R, D)
    sync()
    ref = orc.pool(wave_of(tf, T), P, R, D)
    assert_equal(host(out), ref, "pooled wave")
    assert_equal(host(otf), orc.first_spike(ref), "pooled t_first")


def test_pool_toy_t2(golden):
    g = golden("t2_pool.txt")
    T = int(g["T"][0])
    out, otf = spk.spk_pool(dev(wave_of(g["t_first_in"].astype(np.uint8), T)), 2, 2, 0, out_t_first=None)
    sync()
    assert_equal(host(otf), g["t_first_out"].astype(np.uint8), "T2")


# ---------------------------------------------------------------- pointwise inhibition, potentials pooling
@pytest.mark.parametrize("case", [(3, 15, 30, 28, 28), (2, 15, 250, 14, 14), (2, 9, 7, 5, 3), (1, 4, 1, 2, 2),
                                  (2, 15, 200, 4, 4)])
def test_pointwise_inhibition_parity(case):
    B, T, C, H, W = case
    g = synth.rng(700 + C + H, 0)
    tf = synth.times_uniform_or_silent(g, (B, C, H, W), T, 0.5)
    vf = (g.integers(0, 6, (B, C, H, W)) * 0.5).astype(np.float32)  # ties decided by the feature index
    vf[tf >= T] = 0
    pot = g.normal(0, 3, (B, T, C, H, W)).astype(np.float32)
    rt, rv, rp = orc.pointwise_inhibition(tf, vf, T, pot)
    gp = dev(pot)
    ot, ov, ow = spk.spk_pointwise_inhibition(dev(tf), dev(vf), T, out_wave=None, potentials=gp)
    sync()
    assert_equal(host(ot), rt, "t_first")
    assert_equal(host(ov), rv, "v_first")
    assert_equal(host(ow), orc.expand_wave(rt, T), "wave")
    assert_equal(host(gp), rp, "masked potentials")
    # in place, without the optional outputs
    it, iv = dev(tf), dev(vf)
    spk.spk_pointwise_inhibition(it, iv, T, out_t_first=it, out_v_first=iv)
    sync()
    assert_equal(host(it), rt, "t_first in place")
    assert_equal(host(iv), rv, "v_first in place")


# 2x2 windows of stride 2 on widths that are multiples of 4 take 16-byte loads of
# two rows (the 28x28 map; an odd height, whose last row no window covers); the
# rest one output per thread
@pytest.mark.parametrize("case", [(2, 15, 30, 28, 28, 2, 2, 0), (2, 15, 250, 14, 14, 3, 3, 0),
                                  (1, 5, 4, 9, 11, 3, 2, 1), (1, 3, 2, 7, 7, 4, 3, 2), (2, 4, 3, 5, 6, 1, 1, 0),
                                  (2, 3, 5, 9, 12, 2, 2, 0), (1, 2, 3, 6, 10, 2, 2, 0)])
def test_pool_potentials_parity(case):
    B, T, C, H, W, P, R, D = case
    g = synth.rng(800 + P + C, 0)
    pot = (g.integers(-8, 9, (B, T, C, H, W)) * 0.25).astype(np.float32)  # ties, zeros and negatives
    pot[..., 0, 0] = -0.0
    out = spk.spk_pool_potentials(dev(pot), P, R, D)
    sync()
    ref = orc.pool_potentials(pot, P, R, D)
    assert_equal(host(out).view(np.uint32), ref.view(np.uint32), "pooled potentials (bit patterns)")


# ---------------------------------------------------------------- kWTA
# (B, T, C, H, W, k, radius).  Per-position top-k path: the first five, the
# 1x1 and 1x9 maps, (300 maps of 10x10: feature split with the stash) and
# (k = 16); 16-position tiles: (40x300 maps), (k = 20 > 16) and (k = 16 with
# lists beyond LDS); row tiles: test_kwta_large_tiles.
KWTA_CASES = [(4, 15, 30, 28, 28, 5, 3), (3, 15, 250, 14, 14, 8, 1), (6, 15, 200, 4, 4, 1, 0),
              (2, 30, 20, 10, 25, 1, 5), (3, 4, 3, 5, 7, 12, 1), (2, 15, 5, 40, 300, 6, 2),
              (3, 15, 40, 1, 1, 4, 0), (2, 15, 7, 1, 9, 3, 1), (2, 15, 300, 10, 10, 8, 2),
              (2, 15, 64, 6, 6, 16, 1), (2, 15, 30, 12, 12, 20, 1), (2, 15, 20, 30, 40, 16, 0),
              # below 8 images the lists come from a grid of (image, feature split) workgroups;
              # from 8 on from the rounds' own workgroup (1 to 13 feature splits per position)
              (1, 15, 250, 14, 14, 8, 1), (8, 15, 250, 14, 14, 8, 1), (9, 15, 30, 28, 28, 5, 3),
              (8, 15, 64, 6, 6, 10, 1), (8, 15, 7, 3, 5, 3, 1), (8, 15, 40, 8, 12, 11, 2),
              # the rounds keep each position's best key in registers when a thread owns at most
              # 4 positions (256 images: 256 threads, 3 or 4 positions each), else they walk the
              # lists in LDS every round (65x65 maps: 896 threads, up to 5 positions each)
              (256, 15, 30, 28, 28, 5, 3), (2, 15, 2, 65, 65, 1, 3)]


def kwta_inputs(seed, B, T, C, H, W, ties=True):
    g = synth.rng(300 + seed, 0)
    tf = synth.times_uniform_or_silent(g, (B, C, H, W), T, 0.6)
    if ties:
        vf = (g.integers(0, 6, (B, C, H, W)) * 0.5).astype(np.float32)
    else:
        vf = g.uniform(0, 40, (B, C, H, W)).astype(np.float32)
    vf[tf >= T] = 0
    return tf, vf


@pytest.mark.parametrize("case", KWTA_CASES)
@pytest.mark.parametrize("ties", [True, False])
def test_kwta_parity(case, ties):
    B, T, C, H, W, k, r = case
    tf, vf = kwta_inputs(C + H, B, T, C, H, W, ties)
    win, nw = spk.spk_kwta(dev(tf), dev(vf), T, k, r)
    sync()
    rw, rn = orc.kwta(tf, vf, T, k, r)
    assert_equal(host(nw), rn, "n_winners")
    assert_equal(host(win), rw, "winners")


@pytest.mark.parametrize("case", KWTA_CASES[:2] + [(9, 15, 30, 28, 28, 5, 3)])
def test_kwta_unaligned_inputs(case):
    B, T, C, H, W, k, r = case
    tf, vf = kwta_inputs(C + H + 1, B, T, C, H, W, False)
    win, nw = spk.spk_kwta(dev_shifted(tf), dev_shifted(vf), T, k, r)
    sync()
    rw, rn = orc.kwta(tf, vf, T, k, r)
    assert_equal(host(nw), rn, "n_winners")
    assert_equal(host(win), rw, "winners")


def test_kwta_toy_t3_and_silent(golden):
    g = golden("t3_kwta.txt")
    T = int(g["T"][0])
    tf, vf = dev(g["t_first"].astype(np.uint8)), dev(g["v_first"].astype(np.float32))
    for k, r, key in ((2, 0, "win_k2_r0"), (2, 1, "win_k2_r1"), (5, 1, "win_k5_r1")):
        win, nw = spk.spk_kwta(tf, vf, T, k, r)
        sync()
        assert_equal(host(win), g[key].astype(np.int32), key)
    win, nw = spk.spk_kwta(dev(g["tie_t_first"].astype(np.uint8)), dev(g["tie_v_first"].astype(np.float32)), T, 1, 0)
    sync()
    assert_equal(host(win), g["tie_win"].astype(np.int32), "tie")
    silent = np.full((2, 3, 4, 4), 9, np.uint8)
    win, nw = spk.spk_kwta(dev(silent), dev(np.zeros((2, 3, 4, 4), np.float32)), 9, 3, 1)
    sync()
    assert host(nw).tolist() == [0, 0] and (host(win) == -1).all()


def test_kwta_large_tiles():
    # 256 maps of 256x256: several rows per tile, the multi-row recompute path
    B, T, C, H, W, k, r = 1, 64, 256, 256, 256, 32, 4
    g = synth.rng(77, 0)
    tf = synth.times_geometric(g, (B, C, H, W), T, 0.05)
    vf = g.uniform(0, 100, (B, C, H, W)).astype(np.float32)
    vf[tf >= T] = 0
    win, nw = spk.spk_kwta(dev(tf), dev(vf), T, k, r)
    sync()
    rw, rn = orc.kwta(tf, vf, T, k, r)
    assert_equal(host(nw), rn, "n_winners")
    assert_equal(host(win), rw, "winners")


# ---------------------------------------------------------------- encoding
def test_encode_toy_t4(golden):
    # rank-order only: a 1-channel identity filter passes the intensities through
    g = golden("t4_rank.txt")
    I = g["intensity"].astype(np.float32)[0]  # [1,2,3]
    img = np.clip(I * 10, 0, 255).astype(np.uint8)  # positives keep their order and ties
    ident = np.ones((1, 1, 1), np.float32)
    for T in (2, 3):
        wave, tf, inten = spk.spk_encode_latency(dev(img), dev(ident), T, intensities=None)
        sync()
        assert_equal(host(tf), g[f"t_first_T{T}"].astype(np.uint8), f"T{T}")


ENC_CASES = [("dog", 3, 28, 28, 15, 0.0), ("gabor", 2, 160, 250, 30, 0.0), ("dog", 2, 28, 28, 1, 0.0),
             ("dog", 2, 28, 28, 64, 0.0), ("dog", 1, 28, 28, 255, 0.0), ("rand", 2, 19, 23, 15, 3.0),
             ("pos", 2, 40, 50, 15, 0.0), ("pos", 1, 41, 50, 15, 0.0), ("pos", 3, 1, 1, 15, 0.0),
             ("dog", 1, 100, 300, 15, 0.0),  # 13x13 filters on a wide image: bands of rows
             ("float", 3, 28, 28, 15, 0.0),  # general float taps: the sum order decides the bits
             ("float", 2, 9, 13, 30, -0.5),  # ragged width, negative threshold
             ("flat", 2, 40, 40, 15, 0.0),  # all intensities equal: the index decides every rank
             ("edge", 2, 28, 28, 15, 0.0),  # integer filter form near its int32 bound; a zero channel
             ("bound", 2, 20, 24, 15, 0.0),  # one bit past the integer form's bound: the double form
             # the targets' first digits hold 936 and 968 (padded) keys, and 584 and 592: ranked
             # directly, past the 512 of 64-bit keys the rank step once held
             ("pos", 2, 16, 24, 15, 0.0), ("noise", 2, 40, 40, 15, 0.0)]


@pytest.mark.parametrize("case", ENC_CASES)
def test_encode_parity(case):
    kind, B, H, W, T, thr = case
    g = synth.rng(400 + T, 0)
    if kind == "dog":
        img, bank = synth.stroke_images(g, B, H, W), synth.dog_bank()
    elif kind == "gabor":
        img, bank = synth.pink_noise_images(g, B, H, W), synth.gabor_bank()
    elif kind == "noise":
        img, bank = synth.pink_noise_images(g, B, H, W), synth.dog_bank()
    elif kind == "pos":  # 4 positive filters on a noise image: every entry is ranked
        img = g.integers(1, 256, (B, H, W)).astype(np.uint8)
        bank = (g.integers(1, 65, (4, 3, 3)) / 64.0).astype(np.float32)
    elif kind == "float":
        # channels 1 = -0 and 5 = -4 are exact negations (computed once on the GPU); 3 is
        # -2 but for one tap; 4 = -3 although 3 is itself nearly a negation; taps spread
        # over 2^-20..2^2, so partial sums round and only the defined order reproduces them
        img = synth.stroke_images(g, B, H, W) if H >= 8 else g.integers(0, 256, (B, H, W)).astype(np.uint8)
        base = (g.normal(0, 1, (3, 5, 5)) * np.exp2(g.integers(-20, 3, (3, 5, 5)))).astype(np.float32)
        bank = np.stack([base[0], -base[0], base[1], -base[1], base[2], -base[2]])
        bank[3, 2, 2] += np.float32(0.25)
        bank[4] = -bank[3]
        bank[5] = -bank[4]
    elif kind == "edge":
        # taps k / 2^10, |k| < 2^14: exponent 3 + 10 fraction bits = 13 <= 14, and
        # 169 * 255 * 2^14 < 2^31; sums reach ~2^29 on random pixels.  Channel 1 is
        # all zeros, channel 2 the negation of channel 0 (derived)
        img = g.integers(0, 256, (B, H, W)).astype(np.uint8)
        k = g.integers(-16383, 16384, (13, 13))
        k[6, 6] = 16383
        bank = np.stack([k / 1024.0, np.zeros((13, 13)), -k / 1024.0]).astype(np.float32)
    elif kind == "bound":
        # taps k / 2^11, |k| < 2^15, and one tap k = 2^15 (16.0): one bit past the
        # integer form's int16 limit, so the double form
        img = g.integers(0, 256, (B, H, W)).astype(np.uint8)
        k = g.integers(-32767, 32768, (2, 5, 5))
        k[1, 2, 2] = 32768
        bank = (k / 2048.0).astype(np.float32)
    elif kind == "flat":  # a constant image through a 1x1 filter
        img = np.full((B, H, W), 200, np.uint8)
        img[1, :3, :5] = 0
        bank = np.ones((1, 1, 1), np.float32)
    else:
        img = g.integers(0, 256, (B, H, W)).astype(np.uint8)
        bank = (g.integers(-64, 65, (5, 7, 7)) / 64.0).astype(np.float32)
    wave, tf, inten = spk.spk_encode_latency(dev(img), dev(bank), T, thr, intensities=None)
    sync()
    I, rtf, rwave = orc.encode(img, bank, T, thr)
    assert_equal(host(inten), I, "intensities")
    assert_equal(host(tf), rtf, "t_first")
    assert_equal(host(wave), rwave, "wave")


@pytest.mark.parametrize("r,shape", [(0, (3, 6, 28, 28)), (2, (3, 6, 28, 28)), (8, (3, 6, 28, 28)),
                                     (30, (3, 6, 28, 28)), (8, (1, 2, 100, 250)), (3, (2, 1, 37, 5))])
def test_local_normalization_parity(r, shape):
    # (8, 100x250): rows split over several workgroups; general floats, so the fixed order decides
    g = synth.rng(900 + r + shape[2], 0)
    x = np.abs(g.normal(0, 40, shape)).astype(np.float32)
    x[:, :, :4] = 0.0
    out = spk.spk_local_normalization(dev(x), r, 1e-6)
    sync()
    assert_equal(host(out).view(np.uint32), orc.local_normalize(x, r, 1e-6).view(np.uint32), "normalised (bits)")


@pytest.mark.parametrize("shape,T", [((3, 6, 28, 28), 15), ((2, 4, 41, 50), 15), ((2, 2, 5, 7), 30)])
def test_rank_latency_parity(shape, T):
    g = synth.rng(950 + T + shape[1], 0)
    x = (g.integers(-20, 60, shape) * 0.5).astype(np.float32)  # ties and non-positive entries
    wave, tf = spk.spk_rank_latency(dev(x), T)
    sync()
    rtf = orc.rank_latency(x, T)
    assert_equal(host(tf), rtf, "t_first")
    assert_equal(host(wave), orc.expand_wave(rtf, T), "wave")


def test_chain_encode_with_local_normalization():
    # filter -> local normalisation (radius 8, the tutorial's) -> rank-order code, against the oracle's steps
    from paper_1903_02440_amd.pipeline import chain_for
    wl = synth.mnist_single(4)
    inp = synth.make_inputs(wl)
    ch = chain_for(wl, inp["bank"], local_norm=(8, 1e-12))
    ch.set_weights([torch.from_numpy(w) for w in inp["weights"]])
    ch.set_input(image=torch.from_numpy(inp["image"]))
    ch.forward()
    sync()
    I = orc.filter_images(inp["image"], inp["bank"], 0.0)
    rtf = orc.rank_latency(orc.local_normalize(I, 8, 1e-12), wl.T)
    assert_equal(host(ch.input_tf), rtf, "t_first")
    assert_equal(host(ch.input_wave), orc.expand_wave(rtf, wl.T), "wave")


def test_encode_blank_image_never_spikes():
    img = np.zeros((2, 28, 28), np.uint8)
    wave, tf, _ = spk.spk_encode_latency(dev(img), dev(synth.dog_bank()), 15)
    sync()
    assert (host(tf) == 15).all() and not host(wave).any()


def test_expand_and_validate():
    g = synth.rng(9, 0)
    tf = synth.times_uniform_or_silent(g, (3, 5, 7, 9), 11, 0.3)
    wave = spk.spk_expand_wave(dev(tf), 11)
    bad = spk.spk_validate_wave(wave)
    sync()
    assert_equal(host(wave), orc.expand_wave(tf, 11), "expand")
    assert bad.item() == 0
    w2 = host(wave).copy()
    w2[0, 10, 0, 0, 0] = 0 if w2[0, 9, 0, 0, 0] else w2[0, 10, 0, 0, 0]
    w2[1, 0, 1, 1, 1] = 3
    bad = spk.spk_validate_wave(dev(w2))
    sync()
    assert bad.item() == orc.count_invalid(w2)


# ---------------------------------------------------------------- plasticity
def layer_case(seed, B, T, Cin, H, W, Cout, K, pad, thr, k, r):
    g = synth.rng(500 + seed, 0)
    wave = wave_of(synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5), T)
    Wt = synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05)
    _, _, tf, vf = orc.conv_fire(wave, Wt, pad, thr)
    win, nw = orc.kwta(tf, vf, T, k, r)
    return wave, Wt, win, nw


STDP_CASES = [(1, 8, 15, 6, 28, 28, 30, 5, 2, 15.0, 5, 3), (2, 4, 15, 30, 14, 14, 250, 3, 1, 10.0, 8, 1),
              (3, 6, 15, 250, 4, 4, 200, 5, 2, math.inf, 1, 0)]


@pytest.mark.parametrize("case", STDP_CASES)
def test_stdp_parity(case):
    wave, Wt, win, nw = layer_case(*case)
    pad = case[8]
    Wg = dev(Wt)
    spk.spk_stdp(Wg, pad, dev(wave), dev(win), dev(nw), 0.004, -0.003)
    sync()
    assert_equal(host(Wg), orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003), "weights")


@pytest.mark.parametrize("case", STDP_CASES)
@pytest.mark.parametrize("images", ["batch", "one"])
def test_stdp_first_spike_input(case, images):
    # the layer input given by its first-spike map: the same updates as Eq.4 on its wave
    wave, Wt, win, nw = layer_case(*case)
    if images == "one":
        wave, win, nw = wave[:1], win[:1], nw[:1]
    T, pad = wave.shape[1], case[8]
    tf = orc.first_spike(wave)
    Wg = dev(Wt)
    spk.spk_stdp_first_spike(Wg, pad, dev(tf), T, dev(win), dev(nw), 0.004, -0.003)
    torch.cuda.synchronize()
    assert_equal(host(Wg), orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003), "STDP weights")
    reward = synth.rng(560, 0).choice(np.array([1, -1, 0], np.int8), wave.shape[0])
    Wg = dev(Wt)
    spk.spk_rstdp_first_spike(Wg, pad, dev(tf), T, dev(win), dev(nw), dev(reward), 0.004, -0.003)
    torch.cuda.synchronize()
    assert_equal(host(Wg), orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003, reward=reward), "R-STDP weights")


@pytest.mark.parametrize("case", STDP_CASES)
@pytest.mark.parametrize("rew", [None, 1, -1, 0])
def test_stdp_single_image(case, rew):
    # one image (the online step's direct update): oracle parity for STDP and R-STDP
    wave, Wt, win, nw = layer_case(*case)
    wave, win, nw = wave[:1], win[:1], nw[:1]
    pad = case[8]
    Wg = dev(Wt)
    if rew is None:
        spk.spk_stdp(Wg, pad, dev(wave), dev(win), dev(nw), 0.004, -0.003)
        ref = orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003)
    else:
        reward = np.array([rew], np.int8)
        spk.spk_rstdp(Wg, pad, dev(wave), dev(win), dev(nw), dev(reward), 0.004, -0.003)
        ref = orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003, reward=reward)
    sync()
    assert_equal(host(Wg), ref, "weights")


def test_stdp_single_image_odd_records_match_replay():
    # records the replay skips (a repeated feature, a step outside [0, T), a feature
    # out of range): the one-image path applies the same updates as the batched
    # replay of a two-image batch whose second image has no winners
    wave, Wt, win, nw = layer_case(*STDP_CASES[0])
    T, pad, k = wave.shape[1], 2, win.shape[1]
    w1 = win[:1].copy()
    w1[0, 1] = w1[0, 0]                    # the first record's feature again, other step and place
    w1[0, 1, 1] = (w1[0, 0, 1] + 3) % T
    w1[0, 1, 2:] = (5, 7)
    w1[0, 2, 1] = T                        # a step outside [0, T)
    w1[0, 3, 0] = 999                      # a feature out of range
    n1 = np.array([k], np.int32)
    wave2 = np.concatenate([wave[:1], wave[1:2]])
    win2 = np.concatenate([w1, np.full_like(w1, -1)])
    n2 = np.array([k, 0], np.int32)
    for rates in [(0.004, -0.003), (0.6, -0.5)]:
        Wa, Wb = dev(Wt), dev(Wt)
        spk.spk_stdp(Wa, pad, dev(wave[:1]), dev(w1), dev(n1), *rates)
        spk.spk_stdp(Wb, pad, dev(wave2), dev(win2), dev(n2), *rates)
        sync()
        assert_equal(host(Wa), host(Wb), f"one image vs replay, rates {rates}")


def test_rstdp_and_bounds_variant():
    wave, Wt, win, nw = layer_case(*STDP_CASES[2])
    B = wave.shape[0]
    reward = np.array([1, -1, 0, -1, 1, 1], np.int8)[:B]
    Wg = dev(Wt)
    spk.spk_rstdp(Wg, 2, dev(wave), dev(win), dev(nw), dev(reward), 0.004, -0.003)
    sync()
    assert_equal(host(Wg), orc.stdp(Wt, wave, 2, win, nw, 0.004, -0.003, reward=reward), "R-STDP")
    # stabilizer off, bounds [0.2, 0.8] (the tutorial's variant for its last layer)
    Wg = dev(Wt)
    spk.spk_rstdp(Wg, 2, dev(wave), dev(win), dev(nw), dev(reward), 0.05, -0.04, 0.2, 0.8, stabilizer=False)
    sync()
    ref = orc.stdp(Wt, wave, 2, win, nw, 0.05, -0.04, 0.2, 0.8, stabilizer=False, reward=reward)
    assert_equal(host(Wg), ref, "R-STDP clamp")


@pytest.mark.parametrize("rates", [(0.004, -0.003), (0.7, -0.6)])
def test_stdp_weights_outside_bounds(rates):
    # the first update of a chain starts from a weight outside [lb, ub]; with small
    # rates the later updates skip the clamp, with large ones they keep it
    wave, Wt, win, nw = layer_case(*STDP_CASES[0])
    Wt = Wt.copy()
    g = synth.rng(650, 0)
    flat = Wt.reshape(-1)
    idx = g.choice(flat.size, flat.size // 4, replace=False)
    flat[idx] = g.choice(np.array([-0.25, 1.5, 0.0, 1.0, -0.0], np.float32), idx.size)
    Wg = dev(Wt)
    spk.spk_stdp(Wg, 2, dev(wave), dev(win), dev(nw), *rates)
    sync()
    assert_equal(host(Wg), orc.stdp(Wt, wave, 2, win, nw, *rates), "weights")


def test_stdp_ordered_replay_many_images():
    # more images than one scan chunk, features winning repeatedly: order matters
    g = synth.rng(600, 0)
    B, T, Cin, H, W, Cout, K, pad, k = 2500, 5, 2, 6, 6, 4, 3, 1, 2
    wave = wave_of(synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5), T)
    Wt = synth.normal_weights(g, (Cout, Cin, K, K), 0.5, 0.2)
    win = np.full((B, k, 4), -1, np.int32)
    nw = g.integers(0, k + 1, B).astype(np.int32)
    for b in range(B):
        fs = g.choice(Cout, size=nw[b], replace=False)
        for j, f in enumerate(fs):
            win[b, j] = (f, g.integers(0, T), g.integers(0, H), g.integers(0, W))
    Wg = dev(Wt)
    spk.spk_stdp(Wg, pad, dev(wave), dev(win), dev(nw), 0.02, -0.015)
    sync()
    assert_equal(host(Wg), orc.stdp(Wt, wave, pad, win, nw, 0.02, -0.015), "weights")


def test_decide_parity():
    g = synth.rng(700, 0)
    B, k = 1500, 1
    win = np.full((B, k, 4), -1, np.int32)
    nw = (g.random(B) < 0.9).astype(np.int32)
    win[nw == 1, 0, 0] = g.integers(0, 200, (nw == 1).sum())
    labels = synth.labels(g, B)
    dec, rew = spk.spk_decide(dev(win), dev(nw), dev(labels), 10)
    sync()
    rd, rr = orc.decide(win, nw, labels, 10)
    assert_equal(host(dec), rd, "decision")
    assert_equal(host(rew), rr, "reward")
