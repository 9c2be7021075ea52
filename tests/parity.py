"""Comparison rules shared by the GPU parity tests.

* Integer / byte / index results (spikes, first-spike times, pooled waves,
  winners, encodings): bit-exact.
* Potentials and weights: |gpu - oracle| <= RTOL * |oracle| (so an exact 0
  must be 0).  RTOL = 1e-5.
* A neuron is near-threshold when some step's oracle potential lies within
  RTOL * threshold of the threshold; its spikes / first-spike time / v_first
  are excluded from the exact comparison and counted instead.
"""
import math

import numpy as np

RTOL = 1e-5


def near_threshold_mask(P, thr):
    """[B,Cout,Ho,Wo] mask of neurons with some |P[t] - thr| <= RTOL*thr (P: [B,T,Cout,Ho,Wo])."""
    if math.isinf(thr):
        return np.zeros((P.shape[0],) + P.shape[2:], bool)
    band = RTOL * abs(thr)
    return (np.abs(P.astype(np.float64) - thr) <= band).any(axis=1)


def assert_close(g, o, rtol=RTOL, what=""):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    err = np.abs(g - o)
    bad = err > rtol * np.abs(o)
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside rtol {rtol}; first at {tuple(i)}: "
                             f"gpu {g[tuple(i)]!r} oracle {o[tuple(i)]!r}")


def assert_equal(g, o, what="", mask=None):
    g = np.asarray(g)
    o = np.asarray(o)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    diff = g != o
    if mask is not None:
        diff &= ~mask
    if diff.any():
        i = np.argwhere(diff)[0]
        raise AssertionError(f"{what}: {diff.sum()} of {diff.size} differ; first at {tuple(i)}: "
                             f"gpu {g[tuple(i)]!r} oracle {o[tuple(i)]!r}")


def compare_conv_fire(gpu, orc, thr, exact_potentials=False):
    """gpu / orc: (P, spikes, t_first, v_first) numpy tuples.  Returns the near-threshold count."""
    Pg, Sg, tg, vg = gpu
    Po, So, to, vo = orc
    if exact_potentials:
        assert_equal(Pg, Po, "potentials")
    else:
        assert_close(Pg, Po, what="potentials")
    near = near_threshold_mask(Po, thr)
    assert_equal(tg, to, "t_first", mask=near)
    assert_equal(Sg, So, "spikes", mask=np.broadcast_to(near[:, None], So.shape))
    keep = ~near & (to == tg)
    assert_close(vg[keep], vo[keep], what="v_first")
    return int(near.sum())
