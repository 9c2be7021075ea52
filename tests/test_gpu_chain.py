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


def _near_tie(tf, vf, a, b):
    """Two winner candidates a, b = (f, t, y, x) are tied up to rounding."""
    return a[1] == b[1] and abs(float(vf[a[0], a[2], a[3]]) - float(vf[b[0], b[2], b[3]])) <= \
        RTOL * max(abs(float(vf[a[0], a[2], a[3]])), 1e-30) * 2


def stress_large_small(B=16, HW=32):
    """The large stress layer (64 -> 256 features, 5x5, T = 64, k = 32, r = 4,
    STDP) on HW x HW input maps, small enough for the oracle to run whole."""
    return synth.Workload(5, f"stress-large-{HW}", B, 64, HW, HW, [synth.Conv(64, 256, 5, 2, 40.0, 32, 4)],
                          source="wave", cin=64)


def check_chain(wl, inp, ch, exact, near_log, chunk=16):
    """The GPU chain `ch` (one step done) against the oracle chain, image chunk by
    image chunk (so that the oracle's per-step potentials stay small).

    exact: every output bit-exact, weights included.  Otherwise potentials within
    RTOL, and an image is ambiguous from the first stage where a first-spike time
    differs at a near-threshold neuron or the winners differ at a near tie; the
    features that ambiguous images' winners touch are left out of the weight check.
    Returns the number of ambiguous images."""
    B = wl.B
    keep = [{} for _ in wl.stages]
    dec_all = None
    ambiguous_from = np.full(B, 10 ** 9)
    for c0 in range(0, B, chunk):
        sel = np.arange(c0, min(B, c0 + chunk))
        sl = slice(c0, c0 + len(sel))
        res, src, dec = ochain.forward(wl, inp, inp["weights"], images=sel)
        if dec is not None:
            dec_all = dec if dec_all is None else tuple(np.concatenate([x, y]) for x, y in zip(dec_all, dec))
        if wl.source == "image":
            assert_equal(ch.input_wave[sl].cpu().numpy(), src["wave"], "encoded wave")
        for i, st in enumerate(wl.stages):
            b = ch.bufs[i]
            if hasattr(st, "cout"):
                for k in ("pre_wave", "win", "nw"):
                    keep[i].setdefault(k, []).append(res[i][k])
                P, tf_o = res[i]["P"], res[i]["tf"]
                tf_g = b["tf"][sl].cpu().numpy()
                if exact:
                    assert_equal(b["P"][sl].cpu().numpy(), P, f"stage {i} potentials")
                    assert_equal(b["S"][sl].cpu().numpy(), res[i]["S"], f"stage {i} spikes")
                    assert_equal(tf_g, tf_o, f"stage {i} t_first")
                    assert_equal(b["vf"][sl].cpu().numpy(), res[i]["vf"], f"stage {i} v_first")
                    assert_equal(b["nw"][sl].cpu().numpy(), res[i]["nw"], f"stage {i} n_winners")
                    assert_equal(b["win"][sl].cpu().numpy(), res[i]["win"], f"stage {i} winners")
                    continue
                ok = ambiguous_from[sel] > i
                assert_close(b["P"][sl].cpu().numpy()[ok], P[ok], what=f"stage {i} potentials")
                near = np.zeros(tf_o.shape, bool)
                if not math.isinf(st.thr):
                    near = (np.abs(P.astype(np.float64) - st.thr) <= RTOL * st.thr).any(axis=1)
                wg_all = b["win"][sl].cpu().numpy()
                for j in np.nonzero(ok)[0]:
                    img = sel[j]
                    diff = tf_g[j] != tf_o[j]
                    if diff.any():
                        assert near[j][diff].all(), f"stage {i} image {img}: t_first differs away from threshold"
                        ambiguous_from[img] = i
                        continue
                    wg, wo = wg_all[j], res[i]["win"][j]
                    if not np.array_equal(wg, wo):
                        first = np.nonzero((wg != wo).any(axis=1))[0][0]
                        assert _near_tie(tf_o[j], res[i]["vf"][j], wg[first], wo[first]), \
                            f"stage {i} image {img}: winners differ without a near tie"
                        ambiguous_from[img] = i
            else:
                og = b["out"][sl].cpu().numpy()
                ok = ambiguous_from[sel] > i
                assert_equal(og[ok], res[i]["out"][ok], f"stage {i} pooled wave")
    if dec_all is not None and exact:
        assert_equal(ch.decision.cpu().numpy(), dec_all[0], "decision")
        assert_equal(ch.reward.cpu().numpy(), dec_all[1], "reward")
    full = [{k: np.concatenate(v) for k, v in d.items()} for d in keep]
    new_w = ochain.learn(wl, full, inp["weights"], dec_all)
    n_amb = int((ambiguous_from < 10 ** 9).sum())
    near_log(f"chain {wl.name} B={B} ({'exact' if exact else 'paper'} weights): ambiguous images", n_amb, B)
    for j, (li, gw, ow) in enumerate(zip(conv_idx(wl), ch.weights(), new_w)):
        if exact:
            assert_equal(gw.cpu().numpy(), ow, f"layer {j} weights after plasticity")
            continue
        excl = set()
        for img in np.nonzero(ambiguous_from <= li)[0]:
            for w in (ch.bufs[li]["win"][img].cpu().numpy(), full[li]["win"][img]):
                excl |= set(int(f) for f in w[:, 0] if f >= 0)
        keepf = np.array([f not in excl for f in range(ow.shape[0])])
        if dec_all is not None and wl.stages[li].learn == "rstdp":
            # a changed decision changes the reward sign of every later update of that feature
            bad = ch.decision.cpu().numpy() != dec_all[0]
            for img in np.nonzero(bad)[0]:
                keepf[[int(f) for f in full[li]["win"][img][:, 0] if f >= 0]] = False
        assert_equal(gw.cpu().numpy()[keepf], ow[keepf], f"layer {j} weights (unambiguous features)")
    return n_amb


# the workloads at small batches, and at the batch sizes their benchmark lines run
# (the launch configurations of the conv, kWTA and pooling calls depend on B)
CHAIN_CASES = [(1, 1), (2, 24), (2, 320), (3, 2), (3, 64), (4, 16), (4, 256), ("5s", 16)]


def _workload(wid, B):
    return stress_large_small(B) if wid == "5s" else synth.WORKLOADS[wid](B)


@pytest.mark.parametrize("wid,B", CHAIN_CASES)
def test_chain_bit_exact_with_exact_weights(wid, B, near_log):
    wl = _workload(wid, B)
    inp = synth.make_inputs(wl, weights="dyadic")
    ch = run_gpu(wl, inp)
    check_chain(wl, inp, ch, True, near_log)


@pytest.mark.parametrize("wid,B", CHAIN_CASES)
def test_chain_with_paper_weights(wid, B, near_log):
    wl = _workload(wid, B)
    inp = synth.make_inputs(wl)
    ch = run_gpu(wl, inp)
    n_amb = check_chain(wl, inp, ch, False, near_log)
    assert n_amb <= max(1, B // 4)


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
    features, 5x5) through the chain: sampled potentials / spikes /
    first-spike times against the literal oracle sum (its kWTA and STDP at
    this size: the stage-isolated tests below; the whole layer against the
    oracle: the 32x32-map chain cases)."""
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


def test_full_size_stress_large_kwta():
    """kWTA at the large stress layer's full size (16 images of 256 maps of
    256x256, k = 32, radius 4) on seeded first-spike maps (geometric times, as
    the layer's input) and potentials with ties: winners equal the oracle's
    for all 16 images."""
    B, T, C, H, W, k, r = 16, 64, 256, 256, 256, 32, 4
    g = synth.rng(5, 40)
    tf = synth.times_geometric(g, (B, C, H, W), T, 0.02)
    vf = g.integers(0, 4000, (B, C, H, W), dtype=np.int16).astype(np.float32)
    vf *= np.float32(0.125)
    vf[tf >= T] = 0
    win, nw = spk.spk_kwta(torch.from_numpy(tf).cuda(), torch.from_numpy(vf).cuda(), T, k, r)
    torch.cuda.synchronize()
    print("gpu kWTA done; oracle kWTA over 16 images", flush=True)
    rw, rn = orc.kwta(tf, vf, T, k, r)
    assert_equal(nw.cpu().numpy(), rn, "n_winners")
    assert_equal(win.cpu().numpy(), rw, "winners")
    assert (rn == k).all()


def test_full_size_stress_large_stdp():
    """STDP at the large stress layer's full size: the layer's seeded input
    wave (16 x [64, 64, 256, 256]), its weights, and 32 winners per image with
    distinct features at seeded places (features recur across images, so the
    ordered replay matters): weights equal the oracle's, bit for bit."""
    wl = synth.stress_large()
    inp = synth.make_inputs(wl)
    st = wl.stages[0]
    T = wl.T
    g = synth.rng(5, 41)
    win = np.full((wl.B, st.k, 4), -1, np.int32)
    nw = np.full(wl.B, st.k, np.int32)
    for b in range(wl.B):
        win[b, :, 0] = g.choice(st.cout, st.k, replace=False)
        win[b, :, 1] = g.integers(0, T, st.k)
        win[b, :, 2] = g.integers(0, 256, st.k)
        win[b, :, 3] = g.integers(0, 256, st.k)
    wave = orc.expand_wave(inp["t_first"], T)
    Wg = torch.from_numpy(inp["weights"][0]).cuda()
    spk.spk_stdp(Wg, st.pad, torch.from_numpy(wave).cuda(), torch.from_numpy(win).cuda(),
                 torch.from_numpy(nw).cuda(), st.a_plus, st.a_minus)
    torch.cuda.synchronize()
    ref = orc.stdp(inp["weights"][0], wave, st.pad, win, nw, st.a_plus, st.a_minus)
    assert_equal(Wg.cpu().numpy(), ref, "weights")
    assert not np.array_equal(ref, inp["weights"][0])


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
