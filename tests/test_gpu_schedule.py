"""Learning-rate schedules (section "Tutorial": the full implementation uses
adaptive learning rates and multiplies them over training): rates changed
between steps of the batched chain and of online plasticity, against the
oracle applying the same schedule, bit for bit.

Bit-exact setting: exactly summable initial weights, stabilizer off and
rates that are small powers of two (times 3), so that every weight stays a
multiple of 2^-f and every potential is exact in float over all steps."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle.chain as ochain
import synth
from parity import assert_equal

spk = pytest.importorskip("paper_1903_02440_amd")
from paper_1903_02440_amd.pipeline import chain_for, online_for  # noqa: E402

pytestmark = pytest.mark.gpu

# a doubling schedule with a cap, a+ and a- = -3/4 a+ (the multiplied-rates pattern)
SCHEDULE = [(2.0 ** -9, -3 * 2.0 ** -11), (2.0 ** -8, -3 * 2.0 ** -10), (2.0 ** -7, -3 * 2.0 ** -9),
            (2.0 ** -7, -3 * 2.0 ** -9)]


def exact_workload(B):
    """The tutorial's first layer with the stabilizer off (rates keep the dyadic grid)."""
    st = synth.Conv(6, 30, 5, 2, 15.0, 5, 3, stabilizer=False)
    return synth.Workload(1, "mnist-S1-exact", B, 15, 28, 28, [st], bank="dog")


def test_chain_rates_changed_between_steps():
    wl = exact_workload(16)
    base = synth.make_inputs(wl, weights="dyadic")
    ch = chain_for(wl, base["bank"])
    W = [w.copy() for w in base["weights"]]
    ch.set_weights([torch.from_numpy(w) for w in W])
    g = synth.rng(77, 0)
    for step, (ap, am) in enumerate(SCHEDULE):
        inp = dict(base, image=synth.stroke_images(g, wl.B, wl.H, wl.W))
        ch.set_rates(0, ap, am)
        assert ch.rates(0) == (ap, am)
        ch.set_input(image=torch.from_numpy(inp["image"]), labels=torch.from_numpy(inp["labels"]))
        ch.step()
        torch.cuda.synchronize()
        wl_s = dataclasses.replace(wl, stages=[dataclasses.replace(wl.stages[0], a_plus=ap, a_minus=am)])
        W, res, _ = ochain.step(wl_s, inp, W)
        assert_equal(ch.bufs[0]["win"].cpu().numpy(), res[0]["win"], f"step {step} winners")
        assert_equal(ch.weights()[0].cpu().numpy(), W[0], f"step {step} weights")
    # the workload description itself is untouched by set_rates
    assert (wl.stages[0].a_plus, wl.stages[0].a_minus) == (0.004, -0.003)


def test_online_rates_changed_between_groups():
    wl = exact_workload(24)
    inp = synth.make_inputs(wl, weights="dyadic")
    tr = online_for(wl, inp["bank"], steps_per_graph=4)
    tr.set_weights([torch.from_numpy(w) for w in inp["weights"]])
    W = [w.copy() for w in inp["weights"]]
    imgs = torch.from_numpy(inp["image"]).cuda()
    for grp, (ap, am) in enumerate(SCHEDULE[:3]):
        sel = np.arange(8 * grp, 8 * grp + 8)
        tr.set_rates(0, ap, am)
        tr.run(imgs[sel[0]:sel[-1] + 1])
        torch.cuda.synchronize()
        wl_s = dataclasses.replace(wl, stages=[dataclasses.replace(wl.stages[0], a_plus=ap, a_minus=am)])
        W = ochain.online(wl_s, inp, W, images=sel)[-1]
        assert_equal(tr.weights()[0].cpu().numpy(), W[0], f"group {grp} weights")
