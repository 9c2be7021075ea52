"""CPU oracle for the one-spike-per-neuron convolutional SNN layer.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the
benchmark's CPU-baseline leg are the only callers.  The HIP library never
imports, links or calls anything here, and nothing here touches it.

The arithmetic lives in ``orc.c`` (plain C, double accumulation, one
rounding to float per stored value).  This module compiles it with gcc on
first use (or via :func:`build`) and wraps each entry point with numpy.
Every wrapper states which definition of the paper it follows; the C file
carries the full statement.

Parity status: every function here is pinned by CPU tests in
``tests/test_oracle_*.py`` (hand-computed toys, library special cases,
independent second formulations, invariants and brute force).  The one
quantity with no pin is the whole-network accuracy/timing of the paper's
Table 1, which needs the MNIST data set ("parity unpinned", not claimed).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "orc.c")
_LIB = os.path.join(_HERE, "liborc.so")
# A prebuilt oracle library to load instead (the mutation tests point it at
# deliberately broken copies to show that the pins catch each mistake).
_LIB_OVERRIDE = os.environ.get("ORC_LIB")
_lib = None

_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i8p = np.ctypeslib.ndpointer(dtype=np.int8, flags="C_CONTIGUOUS")
_i64 = ctypes.c_int64
_int = ctypes.c_int
_flt = ctypes.c_float


def build(force: bool = True) -> str:
    """Compile orc.c into liborc.so (single-threaded, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
             "-fvisibility=hidden", "-o", tmp, _SRC, "-lm"],
            check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if _LIB_OVERRIDE:
        lib = ctypes.CDLL(_LIB_OVERRIDE)
    elif not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
        lib = ctypes.CDLL(_LIB)
    else:
        lib = ctypes.CDLL(_LIB)
    sig = {
        "orc_expand_wave": (None, [_u8p, _i64, _int, _i64, _u8p]),
        "orc_first_spike": (None, [_u8p, _i64, _int, _i64, _u8p]),
        "orc_count_invalid": (_i64, [_u8p, _i64, _int, _i64]),
        "orc_filter": (None, [_u8p, _i64, _int, _int, _f32p, _int, _int, _flt, _f32p]),
        "orc_rank_latency": (None, [_f32p, _i64, _i64, _int, _u8p]),
        "orc_conv_wave": (None, [_u8p, _i64, _int, _int, _int, _int, _f32p, _int, _int, _int, _int, _f32p]),
        "orc_conv_times": (None, [_u8p, _i64, _int, _int, _int, _int, _f32p, _int, _int, _int, _int, _f32p]),
        "orc_conv_points": (None, [_u8p, _i64, _int, _int, _int, _int, _f32p, _int, _int, _int, _int,
                                   _i32p, _i64, _f32p]),
        "orc_fire": (None, [_f32p, _i64, _int, _i64, _flt, _int, _u8p, _u8p, _f32p]),
        "orc_pool": (None, [_u8p, _i64, _int, _int, _int, _int, _int, _int, _int, _u8p]),
        "orc_kwta": (None, [_u8p, _f32p, _i64, _int, _int, _int, _int, _int, _int, _i32p, _i32p]),
        "orc_decide": (None, [_i32p, _i32p, _i64, _int, _i32p, _int, _i32p, _i8p]),
        "orc_count_events": (_i64, [_u8p, _i64, _int, _int, _int, _int, _int, _int, _int, _int]),
        "orc_pool_potentials": (None, [_f32p, _i64, _int, _int, _int, _int, _int, _int, _int, _f32p]),
        "orc_local_normalize": (None, [_f32p, _i64, _int, _int, _int, _int, _flt, _f32p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    # orc_stdp takes a nullable reward pointer: declare it with c_void_p.
    lib.orc_stdp.restype = None
    lib.orc_stdp.argtypes = [_f32p, _int, _int, _int, _int, _int, _u8p, _i64, _int, _int, _int,
                             _i32p, _i32p, _int, ctypes.c_void_p, _flt, _flt, _flt, _flt, _int]
    # orc_pointwise_inhibition takes nullable potentials
    lib.orc_pointwise_inhibition.restype = None
    lib.orc_pointwise_inhibition.argtypes = [_u8p, _f32p, _i64, _int, _int, _i64, _u8p, _f32p, ctypes.c_void_p]
    _lib = lib
    return lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---------------------------------------------------------------- Eq.1
def expand_wave(t_first: np.ndarray, T: int) -> np.ndarray:
    """Eq.1: cumulative binary wave [B,T,...] from first-spike times [B,...]."""
    tf = _c(t_first, np.uint8)
    B = tf.shape[0]
    N = tf.size // B if B else 0
    out = np.empty((B, T) + tf.shape[1:], np.uint8)
    _load().orc_expand_wave(tf, B, T, N, out)
    return out


def first_spike(wave: np.ndarray) -> np.ndarray:
    """First step at which each neuron's wave entry is 1 (T if never)."""
    w = _c(wave, np.uint8)
    B, T = w.shape[:2]
    N = w.size // (B * T) if B * T else 0
    out = np.empty((B,) + w.shape[2:], np.uint8)
    _load().orc_first_spike(w, B, T, N, out)
    return out


def count_invalid(wave: np.ndarray) -> int:
    """Neurons whose wave entries are not binary or not non-decreasing in t."""
    w = _c(wave, np.uint8)
    B, T = w.shape[:2]
    N = w.size // (B * T) if B * T else 0
    return int(_load().orc_count_invalid(w, B, T, N))


# ---------------------------------------------------------------- encoding
def filter_images(img: np.ndarray, filt: np.ndarray, thr: float = 0.0) -> np.ndarray:
    """Same-size DoG/Gabor cross-correlation of u8 images, then threshold."""
    im = _c(img, np.uint8)
    fl = _c(filt, np.float32)
    B, H, W = im.shape
    C, KF, _ = fl.shape
    out = np.empty((B, C, H, W), np.float32)
    _load().orc_filter(im, B, H, W, fl, C, KF, float(thr), out)
    return out


def local_normalize(inten: np.ndarray, radius: int, eps: float = 1e-12) -> np.ndarray:
    """Intensities [B,C,H,W] divided by their per-channel regional mean (window
    2r+1, zero padding) plus eps, in a fixed operation order (see orc.c)."""
    x = _c(inten, np.float32)
    B, C, H, W = x.shape
    out = np.empty_like(x)
    _load().orc_local_normalize(x, B, C, H, W, radius, eps, out)
    return out


def rank_latency(inten: np.ndarray, T: int) -> np.ndarray:
    """Rank-order intensity-to-latency: bin floor(rho*T/n) per image."""
    I = _c(inten, np.float32)
    B = I.shape[0]
    N = I.size // B if B else 0
    out = np.empty(I.shape, np.uint8)
    _load().orc_rank_latency(I, B, N, T, out)
    return out


def encode(img: np.ndarray, filt: np.ndarray, T: int, thr: float = 0.0):
    """Image -> (intensities, first-spike times, wave)."""
    I = filter_images(img, filt, thr)
    tf = rank_latency(I, T)
    return I, tf, expand_wave(tf, T)


# ---------------------------------------------------------------- conv / fire
def out_size(n: int, pad: int, K: int, stride: int = 1) -> int:
    """Eq.2 applied to the zero-padded input, floor((n + 2 pad - K) / stride) + 1."""
    return (n + 2 * pad - K) // stride + 1


def conv_wave(wave: np.ndarray, weight: np.ndarray, pad: int, stride: int = 1) -> np.ndarray:
    """Potentials [B,T,Cout,Ho,Wo]: per-step cross-correlation of the wave
    (output (y, x) reads the padded window at (y*stride, x*stride))."""
    w = _c(wave, np.uint8)
    wt = _c(weight, np.float32)
    B, T, Cin, H, W = w.shape
    Cout, Cin2, K, _ = wt.shape
    assert Cin2 == Cin
    Ho, Wo = out_size(H, pad, K, stride), out_size(W, pad, K, stride)
    out = np.empty((B, T, Cout, Ho, Wo), np.float32)
    _load().orc_conv_wave(w, B, T, Cin, H, W, wt, Cout, K, pad, stride, out)
    return out


def conv_times(t_first: np.ndarray, T: int, weight: np.ndarray, pad: int, stride: int = 1) -> np.ndarray:
    """Same potentials from first-spike times (running sum over t)."""
    tf = _c(t_first, np.uint8)
    wt = _c(weight, np.float32)
    B, Cin, H, W = tf.shape
    Cout, Cin2, K, _ = wt.shape
    assert Cin2 == Cin
    Ho, Wo = out_size(H, pad, K, stride), out_size(W, pad, K, stride)
    out = np.empty((B, T, Cout, Ho, Wo), np.float32)
    _load().orc_conv_times(tf, B, T, Cin, H, W, wt, Cout, K, pad, stride, out)
    return out


def conv_points(wave: np.ndarray, weight: np.ndarray, pad: int, pts: np.ndarray, stride: int = 1) -> np.ndarray:
    """Potentials P[b, :, f, y, x] for each row (b, f, y, x) of pts -> [n, T]."""
    w = _c(wave, np.uint8)
    wt = _c(weight, np.float32)
    p = _c(pts, np.int32).reshape(-1, 4)
    B, T, Cin, H, W = w.shape
    Cout, _, K, _ = wt.shape
    out = np.empty((p.shape[0], T), np.float32)
    _load().orc_conv_points(w, B, T, Cin, H, W, wt, Cout, K, pad, stride, p, p.shape[0], out)
    return out


def fire(pot: np.ndarray, thr: float):
    """Threshold firing; thr = +inf selects the in-place Eq.5 mode.

    Returns (potentials, spikes, t_first, v_first); potentials is a copy,
    zeroed before the last step in the Eq.5 mode."""
    P = np.array(pot, dtype=np.float32, order="C", copy=True)
    B, T = P.shape[:2]
    N = P.size // (B * T) if B * T else 0
    spk = np.empty(P.shape, np.uint8)
    tf = np.empty((B,) + P.shape[2:], np.uint8)
    vf = np.empty((B,) + P.shape[2:], np.float32)
    inf_mode = int(np.isinf(thr) and thr > 0)
    _load().orc_fire(P, B, T, N, float(0.0 if inf_mode else thr), inf_mode, spk, tf, vf)
    return P, spk, tf, vf


def conv_fire(wave: np.ndarray, weight: np.ndarray, pad: int, thr: float, stride: int = 1):
    """conv_wave followed by fire: (potentials, spikes, t_first, v_first)."""
    return fire(conv_wave(wave, weight, pad, stride), thr)


# ---------------------------------------------------------------- pool
def pool_size(n: int, P: int, R: int, D: int) -> int:
    """Eq.3 read as floor((n + 2D - P)/R) + 1 (equal to the printed form when P == R)."""
    return (n + 2 * D - P) // R + 1


def pool(wave: np.ndarray, P: int, R: int | None = None, D: int = 0) -> np.ndarray:
    """Spike max-pooling of a wave [B,T,C,H,W] (earliest spike per window)."""
    R = P if R is None else R
    w = _c(wave, np.uint8)
    B, T, C, H, W = w.shape
    out = np.empty((B, T, C, pool_size(H, P, R, D), pool_size(W, P, R, D)), np.uint8)
    _load().orc_pool(w, B, T, C, H, W, P, R, D, out)
    return out


def pool_potentials(pot: np.ndarray, P: int, R: int | None = None, D: int = 0) -> np.ndarray:
    """Max-pooling of potentials [B,T,C,H,W] (largest potential per window; zero padding)."""
    R = P if R is None else R
    x = _c(pot, np.float32)
    B, T, C, H, W = x.shape
    out = np.empty((B, T, C, pool_size(H, P, R, D), pool_size(W, P, R, D)), np.float32)
    _load().orc_pool_potentials(x, B, T, C, H, W, P, R, D, out)
    return out


def pointwise_inhibition(t_first: np.ndarray, v_first: np.ndarray, T: int, potentials: np.ndarray | None = None):
    """Per location only the most salient feature keeps its spike (earliest,
    then highest potential, then lowest feature index): (t_first, v_first)
    [B,C,H,W] of the survivors, and the masked potentials [B,T,C,H,W] if given."""
    tf = _c(t_first, np.uint8)
    vf = _c(v_first, np.float32)
    B, C, H, W = tf.shape
    ot = np.empty_like(tf)
    ov = np.empty_like(vf)
    pot = None if potentials is None else np.array(potentials, dtype=np.float32, order="C", copy=True)
    _load().orc_pointwise_inhibition(tf, vf, B, T, C, H * W, ot, ov,
                                     None if pot is None else pot.ctypes.data_as(ctypes.c_void_p))
    return (ot, ov) if pot is None else (ot, ov, pot)


# ---------------------------------------------------------------- kWTA
def kwta(t_first: np.ndarray, v_first: np.ndarray, T: int, k: int, r: int):
    """Winners [B,k,4] = (f, t, y, x) (-1 padded) and their counts [B]."""
    tf = _c(t_first, np.uint8)
    vf = _c(v_first, np.float32)
    B, C, H, W = tf.shape
    win = np.empty((B, k, 4), np.int32)
    nw = np.empty((B,), np.int32)
    _load().orc_kwta(tf, vf, B, T, C, H, W, k, r, win, nw)
    return win, nw


# ---------------------------------------------------------------- plasticity
def stdp(weight: np.ndarray, pre_wave: np.ndarray, pad: int, winners: np.ndarray,
         n_win: np.ndarray, a_plus: float, a_minus: float, lb: float = 0.0, ub: float = 1.0,
         stabilizer: bool = True, reward: np.ndarray | None = None, stride: int = 1) -> np.ndarray:
    """Eq.4 on the winners (ordered replay over images); returns new weights.

    reward (int8 [B] in {+1,-1,0}) turns it into R-STDP; stride is the
    layer's (the winner (y, x) sees the input window at (y*stride, x*stride))."""
    wt = np.array(weight, dtype=np.float32, order="C", copy=True)
    pw = _c(pre_wave, np.uint8)
    wn = _c(winners, np.int32)
    nw = _c(n_win, np.int32)
    Cout, Cin, K, _ = wt.shape
    B, T, Cin2, H, W = pw.shape
    assert Cin2 == Cin
    k = wn.shape[1]
    rw = None
    if reward is not None:
        rw = _c(reward, np.int8)
        rptr = rw.ctypes.data_as(ctypes.c_void_p)
    else:
        rptr = None
    _load().orc_stdp(wt, Cout, Cin, K, pad, stride, pw, B, T, H, W, wn, nw, k, rptr,
                     float(a_plus), float(a_minus), float(lb), float(ub), int(bool(stabilizer)))
    return wt


def decide(winners: np.ndarray, n_win: np.ndarray, labels: np.ndarray, n_classes: int = 10):
    """Decision (winner feature mod n_classes, -1 silent) and reward (+1/-1/0)."""
    wn = _c(winners, np.int32)
    nw = _c(n_win, np.int32)
    lb = _c(labels, np.int32)
    B, k = wn.shape[:2]
    dec = np.empty((B,), np.int32)
    rew = np.empty((B,), np.int8)
    _load().orc_decide(wn, nw, B, k, lb, n_classes, dec, rew)
    return dec, rew


def count_events(t_first: np.ndarray, T: int, Cout: int, K: int, pad: int, stride: int = 1) -> int:
    """Synaptic events: (spiking pre, post) pairs, each counted once."""
    tf = _c(t_first, np.uint8)
    B, Cin, H, W = tf.shape
    return int(_load().orc_count_events(tf, B, T, Cin, H, W, Cout, K, pad, stride))
