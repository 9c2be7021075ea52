"""Chained parity: whole workloads through the batched HIP chain (the same
Chain class bench.py times) against the oracle chain on the same seeded
inputs.

* Exactly summable ("dyadic") weights make every potential exact in float,
  so the whole chain -- encoding, every layer's spikes / first-spike times /
  winners, pooling, decision and the STDP / R-STDP weights -- must match bit
  for bit.
* With the workloads' own weights, potentials agree within 1e-5 relative and
  a spike can only differ at a neuron whose potential is within 1e-5*theta of
  the threshold; such an image is counted as ambiguous from that layer on and
  the features its winners touched are left out of the weight check.
"""
import math

import numpy as np
import pytest
import torch

import oracle as orc
import oracle.chain as ochain
import synth
from parity import RTOL, assert_close, assert_equal

spk = pytest.importorskip("paper_1903_02440_amd")
from paper_1903_02440_amd.pipeline import chain_for  # noqa: E402

pytestmark = pytest.mark.gpu


def run_gpu(wl, inp):
    ch = chain_for(wl, inp.get("bank"))
    ch.set_weights([torch.from_numpy(w) for w in inp["weights"]])
    lab = torch.from_numpy(inp["labels"])
    if wl.source == "image":
        ch.set_input(image=torch.from_numpy(inp["image"]), labels=lab)
    else:
        ch.set_input(wave=spk.spk_expand_wave(torch.from_numpy(inp["t_first"]).cuda(), wl.T), labels=lab)
    ch.step()
    torch.cuda.synchronize()
    return ch


def gather(X, pts):
    """X[b, :, f, y, x] for each row (b, f, y, x) of pts -> [n, T] on the host."""
    ix = [torch.from_numpy(pts[:, k].astype(np.int64)).cuda() for k in range(4)]
    return X[ix[0], :, ix[1], ix[2], ix[3]].cpu().numpy()


def conv_idx(wl):
    return [i for i, st in enumerate(wl.stages) if hasattr(st, "cout")]


@pytest.mark.parametrize("wid,B", [(1, 1), (2, 24), (3, 2), (4, 16)])
def test_chain_bit_exact_with_exact_weights(wid, B):
    wl = synth.WORKLOADS[wid](B)
    inp = synth.make_inputs(wl, weights="dyadic")
    ch = run_gpu(wl, inp)
    res, src, dec = ochain.forward(wl, inp, inp["weights"])
    if wl.source == "image":
        assert_equal(ch.input_wave.cpu().numpy(), src["wave"], "encoded wave")
    for i, st in enumerate(wl.stages):
        b = ch.bufs[i]
        if hasattr(st, "cout"):
            assert_equal(b["P"].cpu().numpy(), res[i]["P"], f"stage {i} potentials")
            assert_equal(b["S"].cpu().numpy(), res[i]["S"], f"stage {i} spikes")
            assert_equal(b["tf"].cpu().numpy(), res[i]["tf"], f"stage {i} t_first")
            assert_equal(b["vf"].cpu().numpy(), res[i]["vf"], f"stage {i} v_first")
            assert_equal(b["nw"].cpu().numpy(), res[i]["nw"], f"stage {i} n_winners")
            assert_equal(b["win"].cpu().numpy(), res[i]["win"], f"stage {i} winners")
        else:
            assert_equal(b["out"].cpu().numpy(), res[i]["out"], f"stage {i} pooled wave")
    if dec is not None:
        assert_equal(ch.decision.cpu().numpy(), dec[0], "decision")
        assert_equal(ch.reward.cpu().numpy(), dec[1], "reward")
    new_w = ochain.learn(wl, [{k: r[k] for k in ("pre_wave", "win", "nw") if k in r} for r in res],
                         inp["weights"], dec)
    for j, (gw, ow) in enumerate(zip(ch.weights(), new_w)):
        assert_equal(gw.cpu().numpy(), ow, f"layer {j} weights after plasticity")


def _near_tie(tf, vf, a, b):
    """Two winner candidates a, b = (f, t, y, x) are tied up to rounding."""
    return a[1] == b[1] and abs(float(vf[a[0], a[2], a[3]]) - float(vf[b[0], b[2], b[3]])) <= \
        RTOL * max(abs(float(vf[a[0], a[2], a[3]])), 1e-30) * 2


@pytest.mark.parametrize("wid,B", [(1, 1), (2, 32), (3, 2), (4, 16)])
def test_chain_with_paper_weights(wid, B):
    wl = synth.WORKLOADS[wid](B)
    inp = synth.make_inputs(wl)
    ch = run_gpu(wl, inp)
    res, src, dec = ochain.forward(wl, inp, inp["weights"])
    if wl.source == "image":
        assert_equal(ch.input_wave.cpu().numpy(), src["wave"], "encoded wave")
    ambiguous_from = np.full(B, 10 ** 9)  # first stage at which an image became ambiguous
    for i, st in enumerate(wl.stages):
        b = ch.bufs[i]
        ok = ambiguous_from > i
        if hasattr(st, "cout"):
            P = res[i]["P"]
            assert_close(b["P"].cpu().numpy()[ok], P[ok], what=f"stage {i} potentials")
            tf_g, tf_o = b["tf"].cpu().numpy(), res[i]["tf"]
            near = np.zeros(tf_o.shape, bool)
            if not math.isinf(st.thr):
                near = (np.abs(P.astype(np.float64) - st.thr) <= RTOL * st.thr).any(axis=1)
            for img in np.nonzero(ok)[0]:
                diff = tf_g[img] != tf_o[img]
                if diff.any():
                    assert near[img][diff].all(), f"stage {i} image {img}: t_first differs away from threshold"
                    ambiguous_from[img] = i
                    continue
                wg, wo = b["win"].cpu().numpy()[img], res[i]["win"][img]
                if not np.array_equal(wg, wo):
                    vf = res[i]["vf"][img]
                    first = np.nonzero((wg != wo).any(axis=1))[0][0]
                    assert _near_tie(tf_o[img], vf, wg[first], wo[first]), \
                        f"stage {i} image {img}: winners differ without a near tie"
                    ambiguous_from[img] = i
        else:
            og = b["out"].cpu().numpy()
            assert_equal(og[ok], res[i]["out"][ok], f"stage {i} pooled wave")
    n_amb = int((ambiguous_from < 10 ** 9).sum())
    print(f"workload {wid}: {n_amb} of {B} images ambiguous")
    assert n_amb <= max(1, B // 4)
    # weights: features touched by an ambiguous image's winners (either side) are excluded
    new_w = ochain.learn(wl, [{k: r[k] for k in ("pre_wave", "win", "nw") if k in r} for r in res],
                         inp["weights"], dec)
    for j, (li, gw, ow) in enumerate(zip(conv_idx(wl), ch.weights(), new_w)):
        excl = set()
        for img in np.nonzero(ambiguous_from <= li)[0]:
            for w in (ch.bufs[li]["win"].cpu().numpy()[img], res[li]["win"][img]):
                excl |= set(int(f) for f in w[:, 0] if f >= 0)
        keep = np.array([f not in excl for f in range(ow.shape[0])])
        if dec is not None and wl.stages[li].learn == "rstdp":
            # a changed decision changes the reward sign of every later update of that feature
            bad = ch.decision.cpu().numpy() != dec[0]
            for img in np.nonzero(bad)[0]:
                keep[[int(f) for f in res[li]["win"][img][:, 0] if f >= 0]] = False
        assert_equal(gw.cpu().numpy()[keep], ow[keep], f"layer {j} weights (unambiguous features)")


# ---------------------------------------------------------------- full size, bench launch configuration
def test_full_size_mnist_3layer_exact():
    """The headline workload at its benchmark batch (1000 images), one step of
    the same Chain bench.py times, with exactly summable weights: first-spike
    maps, v_first, winners, decisions and the weights after STDP / R-STDP
    equal the oracle's for every image; potentials are checked on a sample."""
    wl = synth.mnist_3layer()
    inp = synth.make_inputs(wl, weights="dyadic")
    ch = run_gpu(wl, inp)
    print("gpu step done; oracle forward over 1000 images", flush=True)
    res, dec = ochain.forward_for_learning(wl, inp, inp["weights"], workers=ochain.default_workers(),
                                           keep=("pre_wave", "win", "nw", "tf", "vf"))
    for i in conv_idx(wl):
        b = ch.bufs[i]
        assert_equal(b["tf"].cpu().numpy(), res[i]["tf"], f"stage {i} t_first")
        assert_equal(b["vf"].cpu().numpy(), res[i]["vf"], f"stage {i} v_first")
        assert_equal(b["win"].cpu().numpy(), res[i]["win"], f"stage {i} winners")
        assert_equal(b["nw"].cpu().numpy(), res[i]["nw"], f"stage {i} n_winners")
    assert_equal(ch.decision.cpu().numpy(), dec[0], "decision")
    assert_equal(ch.reward.cpu().numpy(), dec[1], "reward")
    # sampled potentials of every layer against the literal per-neuron sum
    g = np.random.default_rng(5)
    for i in conv_idx(wl):
        st = wl.stages[i]
        P = ch.bufs[i]["P"]
        pts = np.stack([g.integers(0, wl.B, 200), g.integers(0, st.cout, 200),
                        g.integers(0, P.shape[3], 200), g.integers(0, P.shape[4], 200)], 1).astype(np.int32)
        ref = orc.conv_points(res[i]["pre_wave"], inp["weights"][conv_idx(wl).index(i)], st.pad, pts)
        if math.isinf(st.thr):
            ref[:, :-1] = 0
        got = gather(P, pts)
        assert_equal(got, ref, f"stage {i} sampled potentials")
    new_w = ochain.learn(wl, res, inp["weights"], dec)
    for j, (gw, ow) in enumerate(zip(ch.weights(), new_w)):
        assert_equal(gw.cpu().numpy(), ow, f"layer {j} weights")


def test_full_size_stress_large_sampled():
    """The large stress layer at full size (16 x [64,64,256,256] waves, 256
    features, 5x5): sampled potentials / spikes / first-spike times against
    the literal oracle sum, and the winners and STDP checked by properties."""
    wl = synth.stress_large()
    inp = synth.make_inputs(wl)
    st = wl.stages[0]
    ch = run_gpu(wl, inp)
    T = wl.T
    g = np.random.default_rng(6)
    n = 256
    pts = np.stack([g.integers(0, wl.B, n), g.integers(0, st.cout, n), g.integers(0, 256, n),
                    g.integers(0, 256, n)], 1).astype(np.int32)
    pts[:8, 2:] = [[0, 0], [255, 255], [0, 255], [255, 0], [1, 1], [254, 254], [2, 128], [128, 253]]
    # the oracle needs only the sampled images' waves
    imgs = np.unique(pts[:, 0])
    wave = orc.expand_wave(inp["t_first"][imgs], T)
    local = pts.copy()
    local[:, 0] = np.searchsorted(imgs, pts[:, 0])
    ref = orc.conv_points(wave, inp["weights"][0], st.pad, local)
    b = ch.bufs[0]
    got = gather(b["P"], pts)
    assert_close(got, ref, what="sampled potentials")
    near = (np.abs(ref.astype(np.float64) - st.thr) <= RTOL * st.thr).any(axis=1)
    spk_ref = (ref >= np.float32(st.thr)).astype(np.uint8)
    got_s = gather(b["S"], pts)
    assert_equal(got_s[~near], spk_ref[~near], "sampled spikes")
    tf_ref = np.where(spk_ref.any(1), spk_ref.argmax(1), T)
    ix = [torch.from_numpy(pts[:, k].astype(np.int64)).cuda() for k in range(4)]
    got_tf = b["tf"][ix[0], ix[1], ix[2], ix[3]].cpu().numpy()
    assert_equal(got_tf[~near], tf_ref[~near], "sampled t_first")
    # kWTA properties on the GPU's own first-spike maps (two images): the greedy order is respected
    win, nw = b["win"].cpu().numpy(), b["nw"].cpu().numpy()
    H = W = 256
    for img in (0, wl.B - 1):
        t_img, v_img = b["tf"][img].cpu().numpy(), b["vf"][img].cpu().numpy()
        allowed = t_img < T
        for r in range(nw[img]):
            f, t, y, x = win[img, r]
            assert t_img[f, y, x] == t and allowed[f, y, x]
            cand = np.nonzero(allowed)
            tmin = t_img[cand].min()
            assert t == tmin, "winner is not among the earliest remaining spikes"
            sel = allowed & (t_img == tmin)
            vmax = v_img[sel].max()
            assert v_img[f, y, x] == vmax
            first = np.flatnonzero((sel & (v_img == vmax)).ravel())[0]
            assert first == (f * H + y) * W + x, "tie not broken by the lowest index"
            allowed[f] = False
            allowed[:, max(0, y - st.r):y + st.r + 1, max(0, x - st.r):x + st.r + 1] = False
        if nw[img] < st.k:
            assert not allowed.any()
    # STDP: untouched features keep their weights; touched ones move in Eq.4's direction
    W0 = inp["weights"][0]
    Wn = ch.weights()[0].cpu().numpy()
    used = set(int(f) for f in win[:, :, 0].ravel() if f >= 0)
    for f in range(st.cout):
        if f not in used:
            assert np.array_equal(Wn[f], W0[f])
    assert Wn.min() >= 0 and Wn.max() <= 1


@pytest.mark.parametrize("defer", [False, True])
def test_steps_in_a_row_match_joined_steps(defer):
    # three steps of the 3-layer chain with the plasticity joined at every step end, and
    # with it deferred into the next step (joined before the stage that rewrites each
    # layer's input): identical weights and winners, bit for bit
    wl = synth.WORKLOADS[2](48)
    inp = synth.make_inputs(wl)

    def run(defer_learn):
        ch = chain_for(wl, inp["bank"])
        ch.set_weights([torch.from_numpy(w) for w in inp["weights"]])
        ch.set_input(image=torch.from_numpy(inp["image"]), labels=torch.from_numpy(inp["labels"]))
        for _ in range(3):
            ch.step(defer_learn=defer_learn)
        ch.finish()
        torch.cuda.synchronize()
        return [w.cpu() for w in ch.weights()], [ch.bufs[i]["win"].cpu() for i in ch.conv_stages()]

    w_ref, win_ref = run(False)
    w_got, win_got = run(defer)
    for a, b in zip(w_got, w_ref):
        assert torch.equal(a, b)
    for a, b in zip(win_got, win_ref):
        assert torch.equal(a, b)


def test_compact_chain_matches_full_chain():
    # the compact inter-layer form (no per-step potentials, per-step spikes only where a
    # stage reads them) gives the full chain's first-spike maps, winners, decisions and
    # updated weights, bit for bit
    wl = synth.WORKLOADS[2](40)
    inp = synth.make_inputs(wl)

    def run(compact):
        ch = chain_for(wl, inp["bank"], want_potentials=not compact, want_spikes=not compact)
        ch.set_weights([torch.from_numpy(w) for w in inp["weights"]])
        ch.set_input(image=torch.from_numpy(inp["image"]), labels=torch.from_numpy(inp["labels"]))
        ch.step()
        torch.cuda.synchronize()
        out = [ch.bufs[i][k].cpu() for i in ch.conv_stages() for k in ("tf", "vf", "win", "nw")]
        return out + [w.cpu() for w in ch.weights()] + [ch.decision.cpu(), ch.reward.cpu()]

    for a, b in zip(run(True), run(False)):
        assert torch.equal(a, b)
