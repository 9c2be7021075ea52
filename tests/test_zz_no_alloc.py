"""The allocation-free conv entry point against the workspace one: same
kernels, so bit-identical outputs, on two calls in a row through the C ABI
(the second smaller than the first, so it runs on scratch the first one left
behind)."""
import ctypes
import math

import numpy as np
import pytest
import torch

import synth

spk = pytest.importorskip("paper_1903_02440_amd")

pytestmark = pytest.mark.gpu

# (B, T, Cin, H, W, Cout, K, pad, thr): S2 of the 1000-image workload at 64
# images, then a smaller S1-shaped call; then Eq.5 with a split K (few tasks);
# then Eq.5 in the position-major form (its sums go through the scratch)
CALLS = [[(64, 15, 30, 14, 14, 250, 3, 1, 10.0), (3, 15, 6, 28, 28, 30, 5, 2, 15.0)],
         [(40, 15, 250, 4, 4, 200, 5, 2, math.inf), (2, 15, 250, 4, 4, 200, 5, 2, math.inf)],
         [(300, 15, 250, 4, 4, 200, 5, 2, math.inf), (260, 15, 250, 4, 4, 200, 5, 2, math.inf)]]


def _inputs(seed, B, T, Cin, H, W, Cout, K):
    g = synth.rng(990 + seed, 1)
    tf = torch.from_numpy(synth.times_uniform_or_silent(g, (B, Cin, H, W), T, 0.5)).cuda()
    w = synth.normal_weights(g, (Cout, Cin, K, K), 0.8, 0.05)
    if seed % 2:
        w.reshape(-1)[7] = 1e-12  # the three-term split
    return tf, torch.from_numpy(w).cuda()


def _outputs(B, T, Cout, Ho, Wo):
    return (torch.full((B, T, Cout, Ho, Wo), -7.0, device="cuda"),
            torch.full((B, T, Cout, Ho, Wo), 9, dtype=torch.uint8, device="cuda"),
            torch.full((B, Cout, Ho, Wo), 99, dtype=torch.uint8, device="cuda"),
            torch.full((B, Cout, Ho, Wo), -7.0, device="cuda"))


@pytest.mark.parametrize("calls", CALLS, ids=["finite", "eq5", "eq5-position-major"])
def test_noalloc_matches_workspace_entry(calls):
    lib = spk.lib()
    st = torch.cuda.current_stream().cuda_stream
    for i, (B, T, Cin, H, W, Cout, K, pad, thr) in enumerate(calls):
        tf, w = _inputs(i, B, T, Cin, H, W, Cout, K)
        Ho, Wo = H + 2 * pad - K + 1, W + 2 * pad - K + 1
        got = _outputs(B, T, Cout, Ho, Wo)
        rc = lib.spk_conv_fire_first_spike_noalloc(
            ctypes.c_void_p(tf.data_ptr()), B, T, Cin, H, W, ctypes.c_void_p(w.data_ptr()), Cout, K, pad,
            ctypes.c_float(thr), *[ctypes.c_void_p(x.data_ptr()) for x in got], ctypes.c_void_p(st))
        assert rc == 0, lib.spk_last_error()
        ref = _outputs(B, T, Cout, Ho, Wo)
        spk.spk_conv_fire_first_spike(tf, T, w, pad, thr, *ref)
        torch.cuda.synchronize()
        for a, b, what in zip(got, ref, ("potentials", "spikes", "t_first", "v_first")):
            assert torch.equal(a, b), f"call {i}: {what} differ"
        assert int((got[2] < T).sum()) > 0


def test_noalloc_rejects_calls_beyond_the_scratch():
    # the large stress layer needs ~70 MB of padded input: rejected on the host, nothing launched
    lib = spk.lib()
    buf = torch.zeros(16, dtype=torch.uint8, device="cuda")
    p = ctypes.c_void_p(buf.data_ptr())
    rc = lib.spk_conv_fire_first_spike_noalloc(p, 16, 64, 64, 256, 256, p, 256, 5, 2, ctypes.c_float(40.0),
                                               None, None, p, p, None)
    assert rc == spk.SPK_E_RANGE and b"static scratch" in lib.spk_last_error()
