"""Oracle runs of whole layer chains (test infrastructure, like the rest of
this package): the stages of a workload description applied with the
oracle's functions, in the same order as the batched HIP chain --
frozen-forward over the batch, then the plasticity of every conv stage
replayed image by image."""
from __future__ import annotations

import math
import os

import numpy as np

from . import conv_times, decide, encode, expand_wave, fire, first_spike, kwta, pool, stdp


def _is_conv(st):
    return hasattr(st, "cout")


def _stride(st):
    return getattr(st, "stride", 1)


def forward(wl, inputs, weights, images=None):
    """Per-stage oracle results for the selected images (default: all).

    Returns a list with one dict per stage: conv stages hold pre_wave, P, S,
    tf, vf, win, nw; pool stages hold out.  The source encoding is under
    key "source" of the first dict's parent result (returned as 2nd value),
    and the decision/reward (if the last conv learns by reward) as 3rd."""
    sel = np.arange(wl.B) if images is None else np.asarray(images)
    T = wl.T
    if wl.source == "image":
        I, tf, wave = encode(inputs["image"][sel], inputs["bank"], T)
        src = {"I": I, "tf": tf, "wave": wave}
    else:
        tf = inputs["t_first"][sel]
        wave = expand_wave(tf, T)
        src = {"tf": tf, "wave": wave}
    out = []
    wi = 0
    for st in wl.stages:
        if _is_conv(st):
            P, S, tf1, vf1 = fire(conv_times(tf, T, weights[wi], st.pad, _stride(st)), st.thr)
            win, nw = kwta(tf1, vf1, T, st.k, st.r)
            out.append({"pre_wave": wave, "P": P, "S": S, "tf": tf1, "vf": vf1, "win": win, "nw": nw})
            wave, tf = S, tf1
            wi += 1
        else:
            o = pool(wave, st.P, st.R, st.D)
            out.append({"out": o})
            wave, tf = o, first_spike(o)
    dec = None
    convs = [i for i, st in enumerate(wl.stages) if _is_conv(st)]
    if convs and wl.stages[convs[-1]].learn == "rstdp":
        last = out[convs[-1]]
        dec = decide(last["win"], last["nw"], inputs["labels"][sel], wl.n_classes)
    return out, src, dec


def _fwd_chunk(args):
    wl, inputs, weights, idx, keys = args
    res, _, dec = forward(wl, inputs, weights, idx)
    keep = []
    for r in res:  # only what is asked for, to keep the pipes small
        keep.append({k: v for k, v in r.items() if k in keys})
    return keep, dec


def forward_for_learning(wl, inputs, weights, workers=1, keep=("pre_wave", "win", "nw")):
    """Per-stage results named in `keep` (default: what plasticity needs) and
    the decision/reward of all images, the forward run split over `workers`
    forked processes (the oracle itself stays single-threaded)."""
    chunks = np.array_split(np.arange(wl.B), max(1, workers))
    chunks = [c for c in chunks if len(c)]
    if workers > 1 and len(chunks) > 1:
        import multiprocessing as mp
        with mp.get_context("fork").Pool(len(chunks)) as pool_:
            parts = pool_.map(_fwd_chunk, [(wl, inputs, weights, c, keep) for c in chunks])
    else:
        parts = [_fwd_chunk((wl, inputs, weights, c, keep)) for c in chunks]
    res = []
    for si in range(len(wl.stages)):
        d = {}
        for k in keep:
            vals = [p[0][si][k] for p in parts if k in p[0][si]]
            if vals:
                d[k] = np.concatenate(vals)
        res.append(d)
    dec = None
    if parts[0][1] is not None:
        dec = (np.concatenate([p[1][0] for p in parts]), np.concatenate([p[1][1] for p in parts]))
    return res, dec


def learn(wl, res, weights, dec):
    """New weights after the plasticity of every conv stage (ordered replay)."""
    new = []
    wi = 0
    for st, r in zip(wl.stages, res):
        if not _is_conv(st):
            continue
        W = weights[wi]
        wi += 1
        if st.learn is None:
            new.append(W.copy())
        elif st.learn == "rstdp":
            new.append(stdp(W, r["pre_wave"], st.pad, r["win"], r["nw"], st.a_plus, st.a_minus, st.lb, st.ub,
                            st.stabilizer, reward=dec[1], stride=_stride(st)))
        else:
            new.append(stdp(W, r["pre_wave"], st.pad, r["win"], r["nw"], st.a_plus, st.a_minus, st.lb, st.ub,
                            st.stabilizer, stride=_stride(st)))
    return new


def step(wl, inputs, weights, workers=1):
    """One full pass (forward over the batch, then plasticity): new weights, forward results, decision."""
    res, dec = forward_for_learning(wl, inputs, weights, workers)
    return learn(wl, res, weights, dec), res, dec


def online(wl, inputs, weights, images=None):
    """Online plasticity, one image at a time (section "Tutorial", "Training
    and Testing": each sample's forward runs with the weights the previous
    samples left): `step` on each selected image alone, in order.  Returns
    the weights after every image."""
    import dataclasses
    wl1 = dataclasses.replace(wl, B=1)
    sel = np.arange(wl.B) if images is None else np.asarray(images)
    W = [w.copy() for w in weights]
    after = []
    for i in sel:
        one = dict(inputs)
        one["image"] = inputs["image"][i:i + 1]
        one["labels"] = inputs["labels"][i:i + 1]
        W, _, _ = step(wl1, one, W)
        after.append([w.copy() for w in W])
    return after


def default_workers():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(8, n))


INF = math.inf
