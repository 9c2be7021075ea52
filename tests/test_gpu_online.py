"""Online plasticity (one image per step) on the GPU against the oracle's
sequential one-image steps.

With exactly summable initial weights, the stabilizer off and learning
rates on the weights' dyadic grid (2^-8 and -3*2^-10, near the paper's
0.004 / -0.003), every update is an exact add and the weights stay exactly
summable, so the GPU must match the oracle bit for bit after every image.
With the paper's rates and stabilizer the weights leave that grid; there a
graph-replayed trainer is checked against eager steps of the same trainer.
"""
import dataclasses

import numpy as np
import pytest
import torch

import synth
import oracle.chain as ochain
from paper_1903_02440_amd.pipeline import online_for
from parity import assert_equal

pytestmark = pytest.mark.gpu


def dyadic_online(wl):
    stages = [dataclasses.replace(st, a_plus=2.0 ** -8, a_minus=-3 * 2.0 ** -10, stabilizer=False)
              if hasattr(st, "cout") else st for st in wl.stages]
    return dataclasses.replace(wl, stages=stages)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("make", [synth.mnist_single, synth.mnist_3layer])
def test_online_matches_oracle_after_every_group(make):
    # 9 images in groups of 4: two replays of one captured graph, with host
    # checks between them, then one eager step
    wl = dyadic_online(make(9))
    inp = synth.make_inputs(wl, weights="dyadic")
    ref = ochain.online(wl, inp, inp["weights"])
    tr = online_for(wl, inp["bank"], steps_per_graph=4)
    tr.set_weights([dev(w) for w in inp["weights"]])
    imgs, labs = dev(inp["image"]), dev(inp["labels"])
    for a, b in ((0, 4), (4, 8), (8, 9)):
        print(f"online {wl.name}: images {a}..{b - 1}", flush=True)
        tr.run(imgs[a:b], labs[a:b])
        torch.cuda.synchronize()
        for j, (gw, ow) in enumerate(zip(tr.weights(), ref[b - 1])):
            assert_equal(gw.cpu().numpy(), ow, f"layer {j} weights after image {b - 1}")
    changed = [not np.array_equal(w, w0) for w, w0 in zip(ref[-1], inp["weights"])]
    assert any(changed), "no layer learned"


def test_online_graph_replays_match_eager_steps():
    # the paper's rates and stabilizer: graph replays against eager steps
    wl = synth.mnist_3layer(12)
    inp = synth.make_inputs(wl)
    w0 = [dev(w) for w in inp["weights"]]
    trg = online_for(wl, inp["bank"], steps_per_graph=4)
    tre = online_for(wl, inp["bank"], use_graph=False)
    trg.set_weights(w0)
    tre.set_weights(w0)
    imgs, labs = dev(inp["image"]), dev(inp["labels"])
    for a, b in ((0, 4), (4, 8), (8, 12)):
        print(f"online graph vs eager: images {a}..{b - 1}", flush=True)
        trg.run(imgs[a:b], labs[a:b])
        torch.cuda.synchronize()
        tre.run(imgs[a:b], labs[a:b])
        torch.cuda.synchronize()
        for j, (g, e) in enumerate(zip(trg.weights(), tre.weights())):
            assert_equal(g.cpu().numpy(), e.cpu().numpy(), f"layer {j} weights after image {b - 1}")
    assert any(not torch.equal(g, w) for g, w in zip(trg.weights(), w0)), "no layer learned"
