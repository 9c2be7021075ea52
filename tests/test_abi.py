"""The C ABI: the library loads, exports every symbol the header declares,
and rejects bad arguments on the host before any HIP call -- CPU only."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libspyke.h")

spk = pytest.importorskip("paper_1903_02440_amd")

DUMMY = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation first
DUMMY2 = ctypes.c_void_p(0x2000)


def declared():
    return re.findall(r"^SPK_API\s+[\w\s\*]*?\b(spk_\w+)\s*\(", open(HEADER).read(), flags=re.M)


def test_every_declared_symbol_is_exported():
    names = declared()
    assert len(names) == 34
    lib = spk.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(spk.exported_symbols())


def test_version_and_empty_error():
    assert spk.spk_version() == 0x000100
    assert spk.lib().spk_last_error() in (b"",) or isinstance(spk.lib().spk_last_error(), bytes)


def test_workspace_sizes_are_host_only_and_consistent():
    a = spk.spk_conv_fire_workspace_size(1000, 15, 30, 14, 14, 250, 3, 1)
    b = spk.spk_conv_fire_workspace_size(2000, 15, 30, 14, 14, 250, 3, 1)
    assert 0 < a < b
    assert spk.spk_conv_fire_workspace_size(1, 300, 30, 14, 14, 250, 3, 1) == 0  # T out of range
    assert spk.spk_encode_latency_workspace_size(1000, 6, 28, 28, 15) >= 1000 * 6 * 28 * 28 * 4
    assert spk.spk_kwta_workspace_size(16, 256, 256, 256) == 16 * 4096 * 8
    assert spk.spk_kwta_workspace_size(1, 1, 512, 512) == 0  # H*W above the limit
    # below 8 images the workgroup splits' lists (16 splits of up to 16 keys per position) fit
    assert spk.spk_kwta_workspace_size(1, 250, 14, 14) >= 16 * 196 * 16 * 8
    assert spk.spk_kwta_workspace_size(7, 30, 28, 28) >= 7 * 16 * 784 * 16 * 8
    # the Eq.5 kernel's split partial sums of a small batch are part of the conv workspace
    assert spk.spk_conv_fire_workspace_size(1, 15, 250, 4, 4, 200, 5, 2) >= 25 * 200 * 16 * 4


def _status(fn, *args):
    return fn(*args)


def test_conv_fire_validation_errors():
    lib = spk.lib()
    f = lib.spk_conv_fire
    ok = dict(B=1, T=15, Cin=6, H=28, W=28, Cout=30, K=5, pad=2)

    def call(**kw):
        a = dict(ok, **kw)
        thr = kw.pop("thr", 15.0) if "thr" in kw else 15.0
        return f(DUMMY, a["B"], a["T"], a["Cin"], a["H"], a["W"], DUMMY, a["Cout"], a["K"], a["pad"],
                 a.get("thr", thr), DUMMY, DUMMY, DUMMY, DUMMY, kw.get("ws", DUMMY), kw.get("n", 0), None)

    assert call(T=256) == spk.SPK_E_RANGE
    assert call(T=0) == spk.SPK_E_SHAPE
    assert call(K=40) == spk.SPK_E_SHAPE
    assert call(Cin=3000, K=5) == spk.SPK_E_RANGE
    assert call(n=16) == spk.SPK_E_WORKSPACE
    assert call(thr=float("nan")) == spk.SPK_E_ARG
    assert call(thr=-math.inf) == spk.SPK_E_ARG
    assert b"workspace" in lib.spk_last_error() or b"threshold" in lib.spk_last_error()
    # NULL required outputs
    r = f(DUMMY, 1, 15, 6, 28, 28, DUMMY, 30, 5, 2, 15.0, None, None, None, DUMMY, DUMMY, 1 << 30, None)
    assert r == spk.SPK_E_ARG and b"required" in lib.spk_last_error()


def test_other_validation_errors():
    lib = spk.lib()
    assert lib.spk_pool(DUMMY, 1, 300, 1, 4, 4, 2, 2, 0, DUMMY, None, None) == spk.SPK_E_RANGE
    assert lib.spk_pool(DUMMY, 1, 4, 1, 4, 4, 9, 2, 0, DUMMY, None, None) == spk.SPK_E_SHAPE
    assert lib.spk_pool(None, 1, 4, 1, 4, 4, 2, 2, 0, DUMMY, None, None) == spk.SPK_E_ARG
    assert lib.spk_kwta(DUMMY, DUMMY, 1, 15, 1, 4, 4, 0, 1, DUMMY, DUMMY, DUMMY, 1 << 20, None) == spk.SPK_E_ARG
    assert lib.spk_kwta(DUMMY, DUMMY, 1, 15, 1, 512, 512, 1, 1, DUMMY, DUMMY, DUMMY, 1 << 20, None) == spk.SPK_E_RANGE
    assert lib.spk_kwta(DUMMY, DUMMY, 2, 15, 1, 4, 4, 1, 1, DUMMY, DUMMY, DUMMY, 8, None) == spk.SPK_E_WORKSPACE
    ws = spk.spk_stdp_workspace_size(4, 2, 3, 1, 1)
    assert ws > 0
    assert lib.spk_stdp(DUMMY, 4, 2, 3, 1, DUMMY, 1, 15, 8, 8, DUMMY, DUMMY, 1, 0.004, -0.003, 0.9, 0.1, 1,
                        DUMMY, ws, None) == spk.SPK_E_ARG  # lb > ub
    assert lib.spk_stdp(DUMMY, 4, 2, 3, 1, DUMMY, 1, 15, 8, 8, DUMMY, DUMMY, 1, float("inf"), -0.003, 0.0, 1.0, 1,
                        DUMMY, ws, None) == spk.SPK_E_ARG
    assert lib.spk_stdp(DUMMY, 4, 2, 3, 1, DUMMY, 1, 15, 8, 8, DUMMY, DUMMY, 1, 0.004, -0.003, 0.0, 1.0, 1,
                        DUMMY, ws - 1, None) == spk.SPK_E_WORKSPACE
    assert lib.spk_rstdp(DUMMY, 4, 2, 3, 1, DUMMY, 1, 15, 8, 8, DUMMY, DUMMY, 1, None, 0.004, -0.003, 0.0, 1.0, 1,
                         DUMMY, ws, None) == spk.SPK_E_ARG
    assert lib.spk_encode_latency(DUMMY, 1, 28, 28, DUMMY, 6, 12, 0.0, 15, DUMMY, DUMMY, None, DUMMY, 1 << 30,
                                  None) == spk.SPK_E_RANGE  # even filter size
    assert lib.spk_encode_latency(DUMMY, 1, 28, 28, DUMMY, 6, 13, 0.0, 15, DUMMY, DUMMY, None, DUMMY, 4,
                                  None) == spk.SPK_E_WORKSPACE
    assert lib.spk_expand_wave(DUMMY, 1, 256, 1, 2, 2, DUMMY, None) == spk.SPK_E_RANGE
    assert lib.spk_decide(DUMMY, DUMMY, 4, 0, DUMMY, 10, DUMMY, DUMMY, None) == spk.SPK_E_SHAPE


def test_zero_batch_is_a_no_op():
    lib = spk.lib()
    # B = 0 returns before any launch or pointer use
    assert lib.spk_conv_fire(None, 0, 15, 6, 28, 28, None, 30, 5, 2, 15.0, None, None, None, None, None, 0,
                             None) == spk.SPK_OK
    assert lib.spk_pool(None, 0, 15, 6, 28, 28, 2, 2, 0, None, None, None) == spk.SPK_OK
    assert lib.spk_kwta(None, None, 0, 15, 6, 28, 28, 5, 3, None, None, None, 0, None) == spk.SPK_OK


def test_variant_op_validation_errors():
    lib = spk.lib()
    # pooling of potentials: window larger than the padded input, NULL buffers
    assert lib.spk_pool_potentials(DUMMY, 1, 4, 1, 4, 4, 9, 2, 0, DUMMY, None) == spk.SPK_E_SHAPE
    assert lib.spk_pool_potentials(DUMMY, 1, 4, 1, 4, 4, 2, 0, 0, DUMMY, None) == spk.SPK_E_SHAPE
    assert lib.spk_pool_potentials(None, 1, 4, 1, 4, 4, 2, 2, 0, DUMMY, None) == spk.SPK_E_ARG
    assert lib.spk_pool_potentials(None, 0, 4, 1, 4, 4, 2, 2, 0, None, None) == spk.SPK_OK
    # pointwise inhibition: T range, required outputs (the optional ones may be NULL)
    assert lib.spk_pointwise_inhibition(DUMMY, DUMMY, 1, 256, 2, 4, 4, DUMMY, DUMMY, None, None, None) == spk.SPK_E_RANGE
    assert lib.spk_pointwise_inhibition(DUMMY, DUMMY, 1, 15, 2, 4, 4, None, DUMMY, None, None, None) == spk.SPK_E_ARG
    assert lib.spk_pointwise_inhibition(None, None, 0, 15, 2, 4, 4, None, None, None, None, None) == spk.SPK_OK
    # local normalisation: NaN eps, in-place call, a window that does not fit in LDS
    assert lib.spk_local_normalization(DUMMY, 1, 2, 8, 8, 2, float("nan"), DUMMY2, None) == spk.SPK_E_ARG
    assert lib.spk_local_normalization(DUMMY, 1, 2, 8, 8, 2, 1e-6, DUMMY, None) == spk.SPK_E_ARG
    assert b"separate" in lib.spk_last_error()
    assert lib.spk_local_normalization(DUMMY, 1, 2, 8, 2000, 64, 1e-6, DUMMY2, None) == spk.SPK_E_RANGE
    assert lib.spk_local_normalization(DUMMY, 1, 2, 8, 8, -1, 1e-6, DUMMY2, None) == spk.SPK_E_RANGE
    # rank-order code: workspace too small, no output
    n = spk.spk_rank_latency_workspace_size(2, 6, 28, 28, 15)
    assert n > 0
    assert lib.spk_rank_latency(DUMMY, 2, 6, 28, 28, 15, DUMMY, DUMMY, DUMMY, n - 1, None) == spk.SPK_E_WORKSPACE
    assert lib.spk_rank_latency(DUMMY, 2, 6, 28, 28, 15, None, None, DUMMY, n, None) == spk.SPK_E_ARG
    assert lib.spk_rank_latency(DUMMY, 2, 6, 28, 28, 256, DUMMY, None, DUMMY, n, None) == spk.SPK_E_RANGE


def test_conv_noalloc_rejects_beyond_its_scratch():
    # host-side size check before any HIP call: the large stress layer's padded input exceeds 64 MiB
    lib = spk.lib()
    rc = lib.spk_conv_fire_first_spike_noalloc(DUMMY, 16, 64, 64, 256, 256, DUMMY2, 256, 5, 2, ctypes.c_float(40.0),
                                               None, None, DUMMY, DUMMY2, None)
    assert rc == spk.SPK_E_RANGE and b"static scratch" in lib.spk_last_error()
    assert spk.spk_conv_fire_workspace_size(16, 64, 64, 256, 256, 256, 5, 2) > (64 << 20)
    assert spk.spk_conv_fire_workspace_size(1000, 15, 30, 14, 14, 250, 3, 1) <= (64 << 20)


def test_strided_entry_points_validate_and_size():
    lib = spk.lib()
    f = lib.spk_conv_fire_strided
    # stride 0, stride above 64, a kernel larger than the padded input: rejected before any HIP call
    assert f(DUMMY, 1, 15, 6, 28, 28, DUMMY, 30, 5, 0, 2, 15.0, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, 1 << 30,
             None) == spk.SPK_E_SHAPE
    assert f(DUMMY, 1, 15, 6, 28, 28, DUMMY, 30, 5, 65, 2, 15.0, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, 1 << 30,
             None) == spk.SPK_E_RANGE
    assert lib.spk_conv_fire_first_spike_strided(DUMMY, 1, 15, 6, 3, 3, DUMMY, 30, 9, 2, 2, 15.0, DUMMY, DUMMY,
                                                 DUMMY, DUMMY, DUMMY, 1 << 30, None) == spk.SPK_E_SHAPE
    assert f(None, 0, 15, 6, 28, 28, None, 30, 5, 2, 2, 15.0, None, None, None, None, None, 0, None) == spk.SPK_OK
    # the workspace of a strided call; stride 1 is the plain call's
    assert spk.spk_conv_fire_strided_workspace_size(8, 15, 6, 28, 28, 30, 5, 1, 2) == \
        spk.spk_conv_fire_workspace_size(8, 15, 6, 28, 28, 30, 5, 2)
    assert spk.spk_conv_fire_strided_workspace_size(8, 15, 6, 28, 28, 30, 5, 2, 2) > 0
    assert spk.spk_conv_fire_strided_workspace_size(8, 15, 6, 28, 28, 30, 5, 0, 2) == 0
    assert spk.conv_out_size(28, 5, 2, 2) == 14 and spk.conv_out_size(13, 7, 3, 4) == 4
    ws = spk.spk_stdp_workspace_size(4, 2, 3, 1, 1)
    assert lib.spk_stdp_strided(DUMMY, 4, 2, 3, 0, 1, DUMMY, 1, 15, 8, 8, DUMMY, DUMMY, 1, 0.004, -0.003, 0.0, 1.0,
                                1, DUMMY, ws, None) == spk.SPK_E_SHAPE
    assert lib.spk_rstdp_strided(DUMMY, 4, 2, 3, 2, 1, DUMMY, 1, 15, 8, 8, DUMMY, DUMMY, 1, None, 0.004, -0.003,
                                 0.0, 1.0, 1, DUMMY, ws, None) == spk.SPK_E_ARG
    assert lib.spk_count_events_strided(DUMMY, 1, 15, 2, 8, 8, 4, 3, 0, 1, DUMMY, None) == spk.SPK_E_SHAPE


def test_fused_layer_validation():
    lib = spk.lib()
    f = lib.spk_conv_fire_pool

    def call(H=28, W=28, K=5, pad=2, thr=15.0, pool=2, ptf=DUMMY, B=1):
        return f(DUMMY if B else None, B, 15, 6, H, W, DUMMY, 30, K, pad, thr, pool, None, None, DUMMY, DUMMY2, ptf,
                 None, DUMMY, 1 << 30, None)

    assert call(thr=math.inf) == spk.SPK_E_ARG          # Eq.5 has no fused form
    assert call(pool=0) == spk.SPK_E_SHAPE
    assert call(pool=29) == spk.SPK_E_SHAPE             # window larger than the 28x28 map
    assert call(W=300, pool=2) == spk.SPK_E_RANGE       # a 2-row band of 300 positions
    assert call(ptf=None) == spk.SPK_E_ARG
    assert call(B=0, ptf=None) == spk.SPK_OK


def test_f32mfma_form_needs_a_finite_threshold():
    lib = spk.lib()
    rc = lib.spk_conv_fire_first_spike_f32mfma(DUMMY, 1, 15, 6, 28, 28, DUMMY2, 30, 5, 2, ctypes.c_float(math.inf),
                                               None, None, DUMMY, DUMMY2, DUMMY, 1 << 30, None)
    assert rc == spk.SPK_E_ARG and b"fp32" in lib.spk_last_error()

