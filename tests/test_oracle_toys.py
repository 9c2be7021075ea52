"""Oracle pins: hand-computed toys (tests/golden) -- CPU only."""
import math

import numpy as np

import oracle as orc


def test_t1_wave_and_potentials(golden):
    g = golden("t1_conv_fire.txt")
    T = int(g["T"][0])
    tf = g["t_first_in"].astype(np.uint8)
    wave = orc.expand_wave(tf, T)
    assert np.array_equal(wave, g["wave_in"].astype(np.uint8))
    assert np.array_equal(orc.first_spike(wave), tf)
    W = g["weight"].astype(np.float32)
    P = orc.conv_wave(wave, W, pad=0)
    assert np.array_equal(P, g["potentials"].astype(np.float32))
    P2 = orc.conv_times(tf, T, W, pad=0)
    assert np.array_equal(P2, g["potentials"].astype(np.float32))
    assert orc.count_events(tf, T, Cout=1, K=3, pad=0) == int(g["events"][0])


def test_t1_fire_threshold_equality(golden):
    g = golden("t1_conv_fire.txt")
    T = int(g["T"][0])
    wave = orc.expand_wave(g["t_first_in"].astype(np.uint8), T)
    W = g["weight"].astype(np.float32)
    _, spk, tf, vf = orc.conv_fire(wave, W, 0, float(g["thr_a"][0]))
    assert np.array_equal(spk, g["spikes_a"].astype(np.uint8))
    assert np.array_equal(tf, g["t_first_a"].astype(np.uint8))
    assert np.array_equal(vf, g["v_first_a"].astype(np.float32))
    _, _, tf, vf = orc.conv_fire(wave, W, 0, float(g["thr_b"][0]))
    assert np.array_equal(tf, g["t_first_b"].astype(np.uint8))
    assert np.array_equal(vf, g["v_first_b"].astype(np.float32))
    _, spk, tf, vf = orc.conv_fire(wave, W, 0, float(g["thr_c"][0]))
    assert np.array_equal(tf, g["t_first_c"].astype(np.uint8)) and spk.sum() == 0 and vf.sum() == 0


def test_t1_infinite_threshold(golden):
    g = golden("t1_conv_fire.txt")
    T = int(g["T"][0])
    wave = orc.expand_wave(g["t_first_in"].astype(np.uint8), T)
    P, spk, tf, vf = orc.conv_fire(wave, g["weight"].astype(np.float32), 0, math.inf)
    assert np.array_equal(P, g["potentials_inf"].astype(np.float32))
    assert np.array_equal(spk, g["spikes_inf"].astype(np.uint8))
    assert np.array_equal(tf, g["t_first_inf"].astype(np.uint8))
    assert vf.item() == np.float32(2.625)


def test_t1_padding_orientation(golden):
    g = golden("t1_conv_fire.txt")
    T = int(g["T"][0])
    tf = g["t_first_in"].astype(np.uint8)
    W = g["weight"].astype(np.float32)
    P = orc.conv_wave(orc.expand_wave(tf, T), W, pad=1)
    assert P.shape == (1, T, 1, 3, 3)
    assert np.array_equal(P[0, :, 0, 0, 0], g["potentials_pad1_00"].astype(np.float32))
    assert np.array_equal(orc.conv_times(tf, T, W, pad=1), P)


def test_t2_pool(golden):
    g = golden("t2_pool.txt")
    T = int(g["T"][0])
    wave = orc.expand_wave(g["t_first_in"].astype(np.uint8), T)
    out = orc.pool(wave, 2, 2, 0)
    assert np.array_equal(orc.first_spike(out), g["t_first_out"].astype(np.uint8))


def test_t3_kwta(golden):
    g = golden("t3_kwta.txt")
    T = int(g["T"][0])
    tf = g["t_first"].astype(np.uint8)
    vf = g["v_first"].astype(np.float32)
    w, n = orc.kwta(tf, vf, T, 2, 0)
    assert n[0] == 2 and np.array_equal(w, g["win_k2_r0"].astype(np.int32))
    w, n = orc.kwta(tf, vf, T, 2, 1)
    assert n[0] == 2 and np.array_equal(w, g["win_k2_r1"].astype(np.int32))
    w, n = orc.kwta(tf, vf, T, 5, 1)
    assert n[0] == 2 and np.array_equal(w, g["win_k5_r1"].astype(np.int32))
    w, n = orc.kwta(g["tie_t_first"].astype(np.uint8), g["tie_v_first"].astype(np.float32), T, 1, 0)
    assert n[0] == 1 and np.array_equal(w, g["tie_win"].astype(np.int32))


def test_t4_rank(golden):
    g = golden("t4_rank.txt")
    I = g["intensity"].astype(np.float32)
    assert np.array_equal(orc.rank_latency(I, 2), g["t_first_T2"].astype(np.uint8))
    assert np.array_equal(orc.rank_latency(I, 3), g["t_first_T3"].astype(np.uint8))


def test_t5_stdp(golden):
    g1 = golden("t1_conv_fire.txt")
    g = golden("t5_stdp.txt")
    T = int(g1["T"][0])
    wave = orc.expand_wave(g1["t_first_in"].astype(np.uint8), T)
    W = g1["weight"].astype(np.float32)
    _, _, tf, vf = orc.conv_fire(wave, W, 0, 1.875)
    win, n = orc.kwta(tf, vf, T, 1, 0)
    assert np.array_equal(win[0, 0], [0, 1, 0, 0])
    Wn = orc.stdp(W, wave, 0, win, n, 0.004, -0.003)
    assert np.array_equal(Wn, g["weight_after"].astype(np.float32))
    Wp = orc.stdp(W, wave, 0, win, n, 0.004, -0.003, reward=np.array([-1], np.int8))
    assert np.array_equal(Wp, g["weight_after_punish"].astype(np.float32))
    W0 = orc.stdp(W, wave, 0, win, n, 0.004, -0.003, reward=np.array([0], np.int8))
    assert np.array_equal(W0, W)
