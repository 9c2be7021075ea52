"""Oracle pins against library special cases, second formulations,
invariants and brute force -- CPU only."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as orc
import synth


def _rand_times(seed, shape, T, p_silent=0.3):
    return synth.times_uniform_or_silent(np.random.default_rng(seed), shape, T, p_silent)


# ---------------------------------------------------------------- Eq.1
def test_fig1_shape_and_roundtrip():
    # Fig.1 caption: 3 feature maps of 2x2 neurons and 4 steps -> a 4x3x2x2 wave.
    tf = np.array([[[[0, 3], [4, 1]], [[2, 2], [4, 0]], [[1, 4], [3, 3]]]], np.uint8)
    wave = orc.expand_wave(tf, 4)
    assert wave.shape == (1, 4, 3, 2, 2)
    assert np.array_equal(wave[0, :, 0, 0, 1], [0, 0, 0, 1])  # spikes at t=3, kept to the end
    assert np.array_equal(wave[0, :, 0, 1, 0], [0, 0, 0, 0])  # never
    assert orc.count_invalid(wave) == 0
    assert np.array_equal(orc.first_spike(wave), tf)
    bad = wave.copy()
    bad[0, 3, 0, 1, 1] = 0  # a 1 followed by a 0 (that neuron spikes at t=1)
    bad[0, 0, 1, 0, 0] = 2  # not binary
    assert orc.count_invalid(bad) == 2


def test_wave_monotone_random():
    tf = _rand_times(1, (3, 5, 7, 6), 11)
    wave = orc.expand_wave(tf, 11)
    assert np.all(np.diff(wave.astype(np.int8), axis=1) >= 0)
    assert np.array_equal(11 - wave.sum(axis=1), tf)


# ---------------------------------------------------------------- conv
@pytest.mark.parametrize("pad,K,Cin,Cout,H,W,T", [(0, 3, 2, 3, 7, 6, 4), (2, 5, 3, 4, 9, 8, 6),
                                                  (1, 3, 1, 1, 5, 5, 3)])
def test_conv_matches_torch_float64_per_step(pad, K, Cin, Cout, H, W, T):
    g = np.random.default_rng(7)
    tf = _rand_times(K * 10 + pad, (2, Cin, H, W), T)
    wave = orc.expand_wave(tf, T)
    Wt = g.uniform(0, 1, (Cout, Cin, K, K)).astype(np.float32)
    P = orc.conv_wave(wave, Wt, pad)
    ref = F.conv2d(torch.from_numpy(wave.reshape(-1, Cin, H, W).astype(np.float64)),
                   torch.from_numpy(Wt.astype(np.float64)), padding=pad)
    ref = ref.numpy().astype(np.float32).reshape(P.shape)
    assert np.array_equal(P, ref)


# Stride > 1 (the paper names it as the next version's feature): torch's
# float64 conv2d with the same stride, and the stride-1 map subsampled.
@pytest.mark.parametrize("pad,K,Cin,Cout,H,W,T,s", [(0, 3, 2, 3, 9, 8, 4, 2), (2, 5, 3, 4, 11, 9, 6, 2),
                                                    (1, 3, 2, 2, 10, 7, 5, 3), (0, 2, 1, 2, 9, 10, 3, 3),
                                                    (3, 7, 2, 3, 13, 12, 4, 4)])
def test_conv_stride_matches_torch_float64_per_step(pad, K, Cin, Cout, H, W, T, s):
    g = np.random.default_rng(17)
    tf = _rand_times(K * 10 + pad + s, (2, Cin, H, W), T)
    wave = orc.expand_wave(tf, T)
    Wt = g.uniform(0, 1, (Cout, Cin, K, K)).astype(np.float32)
    P = orc.conv_wave(wave, Wt, pad, s)
    ref = F.conv2d(torch.from_numpy(wave.reshape(-1, Cin, H, W).astype(np.float64)),
                   torch.from_numpy(Wt.astype(np.float64)), padding=pad, stride=s)
    assert P.shape[-2:] == (orc.out_size(H, pad, K, s), orc.out_size(W, pad, K, s)) == tuple(ref.shape[-2:])
    assert np.array_equal(P, ref.numpy().astype(np.float32).reshape(P.shape))
    # the same sums as the stride-1 potentials at every s-th position
    P1 = orc.conv_wave(wave, Wt, pad)
    assert np.array_equal(P, P1[..., ::s, ::s][..., :P.shape[-2], :P.shape[-1]])
    assert np.array_equal(P, orc.conv_times(tf, T, Wt, pad, s)) or \
        np.max(np.abs(P.astype(np.float64) - orc.conv_times(tf, T, Wt, pad, s))) <= np.max(np.spacing(np.abs(P)))
    pts = np.array([[0, 0, 0, 0], [1, Cout - 1, P.shape[-2] - 1, P.shape[-1] - 1]], np.int32)
    c = orc.conv_points(wave, Wt, pad, pts, s)
    for q, (bb, f, y, x) in enumerate(pts):
        assert np.array_equal(c[q], P[bb, :, f, y, x])


def test_stdp_stride_reduces_to_stride_1():
    # a winner (y, x) of a stride-s layer sees the window of the stride-1
    # neuron (y*s, x*s): the updates are identical
    g = np.random.default_rng(21)
    T, Cin, Cout, K, pad, H, W, s, B, k = 8, 3, 5, 3, 1, 11, 10, 2, 3, 3
    wave = orc.expand_wave(_rand_times(12, (B, Cin, H, W), T, 0.5), T)
    Wt = g.uniform(0.05, 0.95, (Cout, Cin, K, K)).astype(np.float32)
    Ho, Wo = orc.out_size(H, pad, K, s), orc.out_size(W, pad, K, s)
    win = np.full((B, k, 4), -1, np.int32)
    nw = np.array([3, 0, 2], np.int32)
    for b in range(B):
        fs = g.permutation(Cout)[:nw[b]]
        for j in range(nw[b]):
            win[b, j] = (fs[j], g.integers(0, T), g.integers(0, Ho), g.integers(0, Wo))
    win[0, 2, 2:] = (Ho - 1, Wo - 1)  # the last window, partly in the padding
    w1 = win.copy()
    w1[..., 2:] = np.where(win[..., 2:] >= 0, win[..., 2:] * s, -1)
    a = orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003, stride=s)
    assert np.array_equal(a, orc.stdp(Wt, wave, pad, w1, nw, 0.004, -0.003))
    assert not np.array_equal(a, orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003))
    rw = np.array([-1, 1, 0], np.int8)
    assert np.array_equal(orc.stdp(Wt, wave, pad, win, nw, 0.004, -0.003, reward=rw, stride=s),
                          orc.stdp(Wt, wave, pad, w1, nw, 0.004, -0.003, reward=rw))


def test_count_events_stride_brute_force():
    T, Cin, Cout, K, pad, H, W, s = 6, 3, 4, 3, 1, 9, 8, 2
    tf = _rand_times(9, (2, Cin, H, W), T, 0.5)
    e = 0
    for b in range(2):
        for y in range((H + 2 * pad - K) // s + 1):
            for x in range((W + 2 * pad - K) // s + 1):
                for ci in range(Cin):
                    for ky in range(K):
                        for kx in range(K):
                            iy, ix = y * s + ky - pad, x * s + kx - pad
                            if 0 <= iy < H and 0 <= ix < W and tf[b, ci, iy, ix] < T:
                                e += Cout
    assert orc.count_events(tf, T, Cout, K, pad, s) == e


def test_fig2_shapes():
    # Fig.2 caption: one 5x5 input map, 3 steps, a 3x3 valid kernel -> [3,1,3,3] potentials.
    tf = _rand_times(3, (1, 1, 5, 5), 3)
    P = orc.conv_wave(orc.expand_wave(tf, 3), np.ones((1, 1, 3, 3), np.float32), 0)
    assert P.shape == (1, 3, 1, 3, 3)
    assert np.all(np.diff(P, axis=1) >= 0)  # cumulative input -> cumulative potentials


def test_conv_two_formulations_agree_exactly_dyadic():
    g = synth.rng(99, 1)
    T, Cin, Cout, K, pad = 9, 4, 5, 3, 1
    tf = _rand_times(5, (3, Cin, 8, 7), T, 0.4)
    Wt = synth.dyadic_weights(g, (Cout, Cin, K, K), Cin * K * K)
    a = orc.conv_wave(orc.expand_wave(tf, T), Wt, pad)
    b = orc.conv_times(tf, T, Wt, pad)
    assert np.array_equal(a, b)


def test_conv_two_formulations_agree_random():
    g = np.random.default_rng(4)
    T, Cin, Cout, K, pad = 15, 6, 7, 5, 2
    tf = _rand_times(6, (2, Cin, 10, 9), T, 0.5)
    Wt = g.normal(0.8, 0.05, (Cout, Cin, K, K)).astype(np.float32)
    a = orc.conv_wave(orc.expand_wave(tf, T), Wt, pad)
    b = orc.conv_times(tf, T, Wt, pad)
    # double sums in two orders, one rounding each: at most one float ulp apart
    assert np.max(np.abs(a.astype(np.float64) - b)) <= np.max(np.spacing(np.abs(a)))
    pts = np.array([[0, 3, 0, 0], [1, 6, 9, 8], [1, 0, 4, 5]], np.int32)
    c = orc.conv_points(orc.expand_wave(tf, T), Wt, pad, pts)
    for q, (bb, f, y, x) in enumerate(pts):
        assert np.array_equal(c[q], a[bb, :, f, y, x])


def test_conv_zero_and_silent():
    T = 5
    tf = np.full((1, 2, 6, 6), T, np.uint8)  # nothing spikes
    P = orc.conv_wave(orc.expand_wave(tf, T), np.ones((3, 2, 3, 3), np.float32), 1)
    assert not P.any()
    assert orc.count_events(tf, T, 3, 3, 1) == 0


def test_count_events_brute_force():
    T, Cin, Cout, K, pad, H, W = 6, 3, 4, 3, 1, 5, 6
    tf = _rand_times(8, (2, Cin, H, W), T, 0.5)
    e = 0
    for b in range(2):
        for y in range(H + 2 * pad - K + 1):
            for x in range(W + 2 * pad - K + 1):
                for ci in range(Cin):
                    for ky in range(K):
                        for kx in range(K):
                            iy, ix = y + ky - pad, x + kx - pad
                            if 0 <= iy < H and 0 <= ix < W and tf[b, ci, iy, ix] < T:
                                e += Cout
    assert orc.count_events(tf, T, Cout, K, pad) == e


# ---------------------------------------------------------------- fire
def test_fire_invariants():
    g = np.random.default_rng(11)
    T = 12
    tf = _rand_times(12, (2, 3, 9, 9), T, 0.3)
    Wt = g.uniform(0, 1, (4, 3, 3, 3)).astype(np.float32)
    P, spk, t1, v1 = orc.conv_fire(orc.expand_wave(tf, T), Wt, 1, 4.0)
    assert orc.count_invalid(spk) == 0  # non-negative weights -> valid cumulative wave
    assert np.array_equal(orc.first_spike(spk), t1)
    B, _, C, H, W = P.shape
    for b, c, y, x in [(0, 0, 0, 0), (1, 3, 8, 8), (1, 2, 4, 5)]:
        s = P[b, :, c, y, x] >= np.float32(4.0)
        t = int(np.argmax(s)) if s.any() else T
        assert t1[b, c, y, x] == t
        assert v1[b, c, y, x] == (P[b, t, c, y, x] if t < T else 0)
    # Eq.5 mode: zero before the last step, spike = positive last potential
    P2, spk2, t2, v2 = orc.fire(P, math.inf)
    assert not P2[:, :-1].any() and np.array_equal(P2[:, -1], P[:, -1])
    assert np.array_equal(spk2[:, -1], (P[:, -1] > 0).astype(np.uint8)) and not spk2[:, :-1].any()
    assert np.array_equal(t2, np.where(P[:, -1] > 0, T - 1, T).astype(np.uint8))


# ---------------------------------------------------------------- pool
@pytest.mark.parametrize("P,R,D,H,W", [(2, 2, 0, 8, 8), (3, 3, 0, 14, 14), (7, 6, 0, 30, 41),
                                       (3, 2, 1, 9, 10)])
def test_pool_matches_torch_maxpool(P, R, D, H, W):
    T = 7
    tf = _rand_times(P * 100 + H, (2, 3, H, W), T, 0.6)
    wave = orc.expand_wave(tf, T)
    out = orc.pool(wave, P, R, D)
    ref = F.max_pool2d(torch.from_numpy(wave.reshape(-1, 3, H, W).astype(np.float64)), P, R, D)
    assert np.array_equal(out, ref.numpy().astype(np.uint8).reshape(out.shape))
    # earliest spike of the window == min of the first-spike times
    tmin = -F.max_pool2d(-torch.from_numpy(tf.astype(np.float64)), P, R, D).numpy()
    if D == 0:
        assert np.array_equal(orc.first_spike(out), tmin.astype(np.uint8))
    assert out.shape[-2:] == ((H + 2 * D - P) // R + 1, (W + 2 * D - P) // R + 1)


def test_pool_sizes_of_the_workloads():
    assert orc.pool_size(28, 2, 2, 0) == 14 and orc.pool_size(14, 3, 3, 0) == 4
    assert orc.pool_size(160, 7, 6, 0) == 26 and orc.pool_size(250, 7, 6, 0) == 41
    # where window == stride Eq.3's printed floor((H+2D)/R) agrees
    for H in range(4, 40):
        for R in (2, 3, 4):
            assert orc.pool_size(H, R, R, 0) == H // R


# ---------------------------------------------------------------- kWTA
def _kwta_greedy(tf, vf, T, k, r):
    """Second formulation: sort every spiking neuron once by the winner
    order, then scan accepting a neuron unless its map already has a winner
    or it lies within r of an accepted winner."""
    C, H, W = tf.shape
    cand = [(int(tf[c, y, x]), -float(vf[c, y, x]), (c * H + y) * W + x)
            for c in range(C) for y in range(H) for x in range(W) if tf[c, y, x] < T]
    cand.sort()
    out = []
    for t, nv, idx in cand:
        if len(out) == k:
            break
        c, y, x = idx // (H * W), (idx // W) % H, idx % W
        if any(c == o[0] or (abs(y - o[2]) <= r and abs(x - o[3]) <= r) for o in out):
            continue
        out.append((c, t, y, x))
    return out


def test_kwta_bruteforce_small_alphabets():
    g = np.random.default_rng(21)
    for trial in range(300):
        C, H, W = int(g.integers(1, 4)), int(g.integers(1, 5)), int(g.integers(1, 5))
        T = int(g.integers(1, 4))
        tf = g.integers(0, T + 1, (1, C, H, W)).astype(np.uint8)
        vf = g.integers(0, 3, (1, C, H, W)).astype(np.float32) * np.float32(0.5)
        k, r = int(g.integers(1, 5)), int(g.integers(0, 3))
        win, n = orc.kwta(tf, vf, T, k, r)
        ref = _kwta_greedy(tf[0], vf[0], T, k, r)
        assert n[0] == len(ref)
        assert [tuple(w) for w in win[0, :n[0]]] == ref, (trial, C, H, W, T, k, r)
        assert np.all(win[0, n[0]:] == -1)


def test_kwta_invariants_random():
    g = np.random.default_rng(5)
    T = 15
    tf = _rand_times(31, (4, 6, 10, 12), T, 0.5)
    vf = g.uniform(0, 50, tf.shape).astype(np.float32)
    k, r = 7, 2
    win, n = orc.kwta(tf, vf, T, k, r)
    for b in range(4):
        w = win[b, :n[b]]
        assert len(set(w[:, 0])) == len(w)  # one winner per feature map
        for i in range(len(w)):
            assert tf[b, w[i, 0], w[i, 2], w[i, 3]] == w[i, 1] < T
            for j in range(i):
                assert max(abs(w[i, 2] - w[j, 2]), abs(w[i, 3] - w[j, 3])) > r
        # every other spiking neuron is blocked by an earlier winner, or k was reached
        if n[b] < k:
            C, H, W = tf.shape[1:]
            for c in range(C):
                for y in range(H):
                    for x in range(W):
                        if tf[b, c, y, x] < T:
                            assert any(c == o[0] or (abs(y - o[2]) <= r and abs(x - o[3]) <= r) for o in w)


# ---------------------------------------------------------------- encoding
def test_filter_matches_torch_and_zero_on_flat():
    img = synth.stroke_images(synth.rng(1, 0), 3)
    bank = synth.dog_bank()
    I = orc.filter_images(img, bank, -np.inf)
    ref = F.conv2d(torch.from_numpy(img[:, None].astype(np.float64)),
                   torch.from_numpy(bank[:, None].astype(np.float64)), padding=bank.shape[-1] // 2)
    assert np.array_equal(I, ref.numpy().astype(np.float32))
    thr = orc.filter_images(img, bank, 0.0)
    assert np.array_equal(thr, np.where(I < 0, 0, I))
    flat = np.full((1, 20, 20), 255, np.uint8)  # zero-sum bank: interior of a flat region is exactly 0
    If = orc.filter_images(flat, bank, -np.inf)
    assert not If[:, :, 6:14, 6:14].any()
    gab = synth.gabor_bank()
    assert gab.shape == (4, 5, 5) and np.all(gab.sum(axis=(1, 2)) == 0)


def test_rank_latency_invariants_and_bruteforce():
    g = np.random.default_rng(2)
    for trial in range(40):
        T = int(g.integers(1, 20))
        I = g.integers(-3, 6, (2, 3, 4, 5)).astype(np.float32) * np.float32(0.25)  # many ties
        tf = orc.rank_latency(I, T)
        for b in range(2):
            v, t = I[b].ravel(), tf[b].ravel()
            pos = np.nonzero(v > 0)[0]
            n = len(pos)
            assert np.all(t[v <= 0] == T) and np.all(t[pos] < T)
            order = sorted(pos, key=lambda i: (-v[i], i))
            for rho, i in enumerate(order):
                assert t[i] == rho * T // n
            if n:
                counts = np.bincount(t[pos], minlength=T)
                assert set(counts) <= {n // T, -(-n // T)}
                for i in pos:  # larger intensity never spikes later
                    assert np.all(t[pos][v[pos] < v[i]] >= t[i])


# ---------------------------------------------------------------- plasticity
def _layer_case(seed=3, T=10, Cin=3, Cout=5, K=3, pad=1, H=8, W=8, B=4):
    g = np.random.default_rng(seed)
    tf = _rand_times(seed, (B, Cin, H, W), T, 0.4)
    wave = orc.expand_wave(tf, T)
    Wt = g.uniform(0.05, 0.95, (Cout, Cin, K, K)).astype(np.float32)
    P, spk, t1, v1 = orc.conv_fire(wave, Wt, pad, 2.0)
    win, n = orc.kwta(t1, v1, T, 3, 1)
    return wave, Wt, win, n


def test_stdp_fixed_points_and_identity():
    wave, Wt, win, n = _layer_case()
    W2 = Wt.copy()
    W2[..., 0] = 0.0
    W2[..., 1] = 1.0
    Wn = orc.stdp(W2, wave, 1, win, n, 0.004, -0.003)
    assert np.array_equal(Wn[..., :2], W2[..., :2])  # LB and UB are fixed points of Eq.4
    assert np.array_equal(orc.stdp(Wt, wave, 1, win, n, 0.0, 0.0), Wt)
    Wn = orc.stdp(Wt, wave, 1, win, n, 0.004, -0.003)
    used = set(win[:, :, 0][win[:, :, 0] >= 0].tolist())
    for f in range(Wt.shape[0]):
        if f not in used:
            assert np.array_equal(Wn[f], Wt[f])
    assert Wn.min() >= 0 and Wn.max() <= 1
    # bounds and stabilizer off (tutorial variant): plain additive steps, clamped
    Wc = orc.stdp(Wt, wave, 1, win, n, 0.5, -0.5, lb=0.2, ub=0.8, stabilizer=False)
    assert Wc.min() >= np.float32(0.2) and Wc.max() <= np.float32(0.8)


def test_stdp_sign_and_single_step():
    # one winner, direct check of every synapse against Eq.4
    wave, Wt, win, n = _layer_case(seed=9, B=1)
    w1 = win[:, :1].copy()
    n1 = np.minimum(n, 1)
    Wn = orc.stdp(Wt, wave, 1, w1, n1, 0.004, -0.003)
    f, t, y, x = w1[0, 0]
    Cout, Cin, K, _ = Wt.shape
    H, W = wave.shape[-2:]
    for ci in range(Cin):
        for ky in range(K):
            for kx in range(K):
                iy, ix = y + ky - 1, x + kx - 1
                pre = 0 <= iy < H and 0 <= ix < W and wave[0, t, ci, iy, ix] == 1
                w = float(Wt[f, ci, ky, kx])
                a = 0.004 if pre else -0.003
                exp = np.float32(np.clip(w + float(np.float32(a)) * (w * (1 - w)), 0, 1))
                assert Wn[f, ci, ky, kx] == exp
                assert (Wn[f, ci, ky, kx] > Wt[f, ci, ky, kx]) == pre


def test_rstdp_reduces_to_stdp():
    wave, Wt, win, n = _layer_case(seed=4)
    B = wave.shape[0]
    plus = orc.stdp(Wt, wave, 1, win, n, 0.004, -0.003, reward=np.ones(B, np.int8))
    assert np.array_equal(plus, orc.stdp(Wt, wave, 1, win, n, 0.004, -0.003))
    minus = orc.stdp(Wt, wave, 1, win, n, 0.004, -0.003, reward=-np.ones(B, np.int8))
    assert np.array_equal(minus, orc.stdp(Wt, wave, 1, win, n, -0.004, 0.003))
    none = orc.stdp(Wt, wave, 1, win, n, 0.004, -0.003, reward=np.zeros(B, np.int8))
    assert np.array_equal(none, Wt)


def test_stdp_ordered_replay_is_online():
    # batch of B = replay image by image (the per-sample rule for B = 1)
    wave, Wt, win, n = _layer_case(seed=6)
    batch = orc.stdp(Wt, wave, 1, win, n, 0.004, -0.003)
    online = Wt
    for b in range(wave.shape[0]):
        online = orc.stdp(online, wave[b:b + 1], 1, win[b:b + 1], n[b:b + 1], 0.004, -0.003)
    assert np.array_equal(batch, online)
    # within one image the winners use distinct features: their order is irrelevant
    perm = win[:, ::-1].copy()
    for b in range(wave.shape[0]):
        perm[b, :n[b]] = win[b, :n[b]][::-1]
    assert np.array_equal(orc.stdp(Wt, wave, 1, perm, n, 0.004, -0.003), batch)


def test_decide():
    win = np.array([[[13, 14, 0, 1]], [[7, 3, 2, 2]], [[-1, -1, -1, -1]]], np.int32)
    n = np.array([1, 1, 0], np.int32)
    dec, rew = orc.decide(win, n, np.array([3, 5, 0], np.int32), 10)
    assert dec.tolist() == [3, 7, -1] and rew.tolist() == [1, -1, 0]


def test_filter_asymmetric_kernel_orientation():
    # cross-correlation (no flip) and same padding, checked with a non-symmetric bank
    g = np.random.default_rng(17)
    img = g.integers(0, 256, (2, 9, 11)).astype(np.uint8)
    bank = (g.integers(-64, 65, (3, 5, 5)) / 64.0).astype(np.float32)
    I = orc.filter_images(img, bank, -np.inf)
    ref = F.conv2d(torch.from_numpy(img[:, None].astype(np.float64)),
                   torch.from_numpy(bank[:, None].astype(np.float64)), padding=2)
    assert np.array_equal(I, ref.numpy().astype(np.float32))


# ---------------------------------------------------------------- online plasticity
def test_online_composes_one_image_steps():
    """online() is `step` on each image alone, in order: one image equals a
    one-image batch; zero rates leave the weights as they were; the weights
    after image k do not depend on later images; and order matters."""
    import dataclasses
    import oracle.chain as ochain
    wl = synth.mnist_single(3)
    inp = synth.make_inputs(wl)
    after = ochain.online(wl, inp, inp["weights"])
    one = dict(inp, image=inp["image"][:1], labels=inp["labels"][:1])
    W1, _, _ = ochain.step(dataclasses.replace(wl, B=1), one, inp["weights"])
    assert np.array_equal(after[0][0], W1[0])
    first2 = ochain.online(wl, inp, inp["weights"], images=[0, 1])
    assert np.array_equal(first2[1][0], after[1][0])
    rev = ochain.online(wl, inp, inp["weights"], images=[2, 1, 0])
    assert not np.array_equal(rev[2][0], after[2][0])
    still = dataclasses.replace(wl, stages=[dataclasses.replace(wl.stages[0], a_plus=0.0, a_minus=0.0)])
    frozen = ochain.online(still, inp, inp["weights"])
    assert np.array_equal(frozen[-1][0], inp["weights"][0])


# ---------------------------------------------------------------- potentials pooling, pointwise inhibition
@pytest.mark.parametrize("P,R,D", [(2, 2, 0), (3, 3, 0), (3, 2, 1), (4, 3, 2), (1, 1, 0)])
def test_pool_potentials_is_max_pool_of_the_zero_padded_map(P, R, D):
    g = np.random.default_rng(31 + P + R + D)
    x = g.normal(0, 2, (2, 3, 4, 9, 11)).astype(np.float32)
    got = orc.pool_potentials(x, P, R, D)
    xt = F.pad(torch.from_numpy(x).reshape(-1, 1, 9, 11), (D, D, D, D), value=0.0)
    ref = F.max_pool2d(xt, P, R).reshape(got.shape).numpy()
    assert np.array_equal(got, ref)


def test_pointwise_inhibition_second_formulation():
    """Against a lexicographic sort per location: the survivor is the first of
    (t_first, -v_first, feature) among spiking features; everything else is
    silenced, and the masked potentials keep only the survivor's planes."""
    g = np.random.default_rng(5)
    B, T, C, H, W = 3, 9, 7, 4, 5
    tf = np.where(g.random((B, C, H, W)) < 0.4, T, g.integers(0, T, (B, C, H, W))).astype(np.uint8)
    vf = (g.integers(0, 4, (B, C, H, W)) * 0.5).astype(np.float32)  # many ties
    vf[tf >= T] = 0
    pot = g.normal(0, 1, (B, T, C, H, W)).astype(np.float32)
    ot, ov, op = orc.pointwise_inhibition(tf, vf, T, pot)
    for b in range(B):
        for y in range(H):
            for x in range(W):
                spiking = [c for c in range(C) if tf[b, c, y, x] < T]
                win = min(spiking, key=lambda c: (tf[b, c, y, x], -vf[b, c, y, x], c)) if spiking else None
                for c in range(C):
                    keep = c == win
                    assert ot[b, c, y, x] == (tf[b, c, y, x] if keep else T)
                    assert ov[b, c, y, x] == (vf[b, c, y, x] if keep else 0.0)
                    assert np.array_equal(op[b, :, c, y, x], pot[b, :, c, y, x] if keep else np.zeros(T, np.float32))


@pytest.mark.parametrize("r", [0, 1, 3, 8, 40])
def test_local_normalize_against_box_sums(r):
    """Exactly summable intensities (multiples of 1/16 below 2^12): every
    window sum is exact in double whatever the order, so a box sum from a
    padded array and float32 arithmetic reproduce the oracle bit for bit; r = 0
    gives in / (in + eps), and a window beyond the image sees the zero padding."""
    g = np.random.default_rng(40 + r)
    x = (g.integers(0, 1 << 16, (2, 3, 9, 13)) / 16.0).astype(np.float32)
    eps = np.float32(1e-3)
    got = orc.local_normalize(x, r, float(eps))
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (r, r), (r, r)))
    S = np.zeros(x.shape, np.float64)
    for dy in range(2 * r + 1):
        for dx in range(2 * r + 1):
            S += xp[:, :, dy:dy + 9, dx:dx + 13]
    mean = (S / float((2 * r + 1) ** 2)).astype(np.float32)
    ref = x / (mean + eps)
    assert np.array_equal(got, ref)
    if r == 0:
        assert np.array_equal(got, x / (x + eps))
