"""Python binding of libspyke, the gfx950 hot path for convolutional spiking
networks with at most one spike per neuron (Mozafari et al., SpykeTorch, 2019).

Every ``spk_*`` function here has the name of the C entry point it calls
(``include/libspyke.h`` documents the semantics) and only marshals
arguments: it checks dtypes/shapes, allocates the outputs and workspace it
is not given (torch device memory), passes raw pointers plus the current
HIP stream, and raises :class:`SpykeError` on a non-zero status.  All
computation happens in the HIP kernels of ``libspyke.so``; there is no
fallback -- importing fails loudly when the library is missing.

Output arguments accept a tensor (written in place), ``None`` (allocated
here) or ``False`` (the optional output is skipped: NULL is passed).
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspyke.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libspyke.so is not built ({LIB_PATH}); run `python -m paper_1903_02440_amd.build`")

_lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_Z = ctypes.c_size_t

_SIGS = {
    "spk_version": (_I, []),
    "spk_last_error": (ctypes.c_char_p, []),
    "spk_encode_latency_workspace_size": (_Z, [_I, _I, _I, _I, _I]),
    "spk_encode_latency": (_I, [_P, _I, _I, _I, _P, _I, _I, _F, _I, _P, _P, _P, _P, _Z, _P]),
    "spk_expand_wave": (_I, [_P, _I, _I, _I, _I, _I, _P, _P]),
    "spk_rank_latency_workspace_size": (_Z, [_I, _I, _I, _I, _I]),
    "spk_rank_latency": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _Z, _P]),
    "spk_local_normalization": (_I, [_P, _I, _I, _I, _I, _I, _F, _P, _P]),
    "spk_validate_wave": (_I, [_P, _I, _I, _I, _I, _I, _P, _P]),
    "spk_conv_fire_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I, _I]),
    "spk_conv_fire": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _F, _P, _P, _P, _P, _P, _Z, _P]),
    "spk_conv_fire_first_spike": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _F, _P, _P, _P, _P, _P, _Z, _P]),
    "spk_conv_fire_first_spike_noalloc": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _F, _P, _P, _P, _P, _P]),
    "spk_pool": (_I, [_P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P]),
    "spk_pool_first_spike": (_I, [_P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P]),
    "spk_pool_potentials": (_I, [_P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P]),
    "spk_pointwise_inhibition": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "spk_kwta_workspace_size": (_Z, [_I, _I, _I, _I]),
    "spk_kwta": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _Z, _P]),
    "spk_stdp_workspace_size": (_Z, [_I, _I, _I, _I, _I]),
    "spk_stdp": (_I, [_P, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _F, _F, _F, _F, _I, _P, _Z, _P]),
    "spk_rstdp": (_I, [_P, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _P, _F, _F, _F, _F, _I, _P, _Z, _P]),
    "spk_decide": (_I, [_P, _P, _I, _I, _P, _I, _P, _P, _P]),
    "spk_count_events": (_I, [_P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P]),
    "spk_conv_fire_first_spike_f32mfma": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _F, _P, _P, _P, _P, _P, _Z,
                                               _P]),
    "spk_conv_fire_pool": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _F, _I, _P, _P, _P, _P, _P, _P, _P, _Z,
                                _P]),
    "spk_conv_fire_strided_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I, _I, _I]),
    "spk_conv_fire_strided": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _F, _P, _P, _P, _P, _P, _Z, _P]),
    "spk_conv_fire_first_spike_strided": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _F, _P, _P, _P, _P, _P,
                                               _Z, _P]),
    "spk_stdp_first_spike": (_I, [_P, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _F, _F, _F, _F, _I, _P, _Z,
                                  _P]),
    "spk_rstdp_first_spike": (_I, [_P, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _P, _F, _F, _F, _F, _I, _P,
                                   _Z, _P]),
    "spk_stdp_strided": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _F, _F, _F, _F, _I, _P, _Z,
                              _P]),
    "spk_rstdp_strided": (_I, [_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _P, _P, _I, _P, _F, _F, _F, _F, _I, _P,
                               _Z, _P]),
    "spk_count_events_strided": (_I, [_P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

SPK_OK, SPK_E_ARG, SPK_E_SHAPE, SPK_E_RANGE, SPK_E_WORKSPACE, SPK_E_INPUT, SPK_E_HIP = range(7)


class SpykeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libspyke status {status}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded libspyke.so (for callers that marshal pointers themselves)."""
    return _lib


def exported_symbols():
    return list(_SIGS)


def _check(status: int):
    if status != SPK_OK:
        raise SpykeError(status, _lib.spk_last_error().decode())


def _ptr(t):
    if t is None or t is False:
        return None
    if not t.is_contiguous():
        raise ValueError("libspyke needs contiguous tensors")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, dtype, shape, name):
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a device tensor")


def _out(t, shape, dtype, device, name):
    if t is False:
        return False
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _need(t, dtype, shape, name)
    return t


def _ws(ws, nbytes, device):
    if nbytes == 0:
        return None
    if ws is None:
        return torch.empty(nbytes, dtype=torch.uint8, device=device)
    if ws.numel() * ws.element_size() < nbytes:
        raise ValueError(f"workspace needs {nbytes} bytes")
    return ws


def spk_version() -> int:
    return int(_lib.spk_version())


# ---------------------------------------------------------------- encoding
def spk_encode_latency_workspace_size(B, C, H, W, T) -> int:
    return int(_lib.spk_encode_latency_workspace_size(B, C, H, W, T))


def spk_encode_latency(image, filters, T, filter_threshold=0.0, wave=None, t_first=None, intensities=False,
                       workspace=None, stream=None):
    """image u8 [B,H,W], filters f32 [C,KF,KF] -> (wave, t_first, intensities)."""
    B, H, W = image.shape
    C, KF, _ = filters.shape
    _need(image, torch.uint8, (B, H, W), "image")
    _need(filters, torch.float32, (C, KF, KF), "filters")
    dev = image.device
    wave = _out(wave, (B, T, C, H, W), torch.uint8, dev, "wave")
    t_first = _out(t_first, (B, C, H, W), torch.uint8, dev, "t_first")
    intensities = _out(intensities, (B, C, H, W), torch.float32, dev, "intensities")
    n = spk_encode_latency_workspace_size(B, C, H, W, T)
    ws = _ws(workspace, n, dev)
    _check(_lib.spk_encode_latency(_ptr(image), B, H, W, _ptr(filters), C, KF, float(filter_threshold), T,
                                   _ptr(wave), _ptr(t_first), _ptr(intensities), _ptr(ws), n, _stream(stream)))
    return wave, t_first, intensities


def spk_rank_latency_workspace_size(B, C, H, W, T) -> int:
    return int(_lib.spk_rank_latency_workspace_size(B, C, H, W, T))


def spk_rank_latency(intensities, T, wave=None, t_first=None, workspace=None, stream=None):
    """Rank-order code of an intensity map f32 [B,C,H,W] -> (wave u8 [B,T,C,H,W], t_first u8 [B,C,H,W])."""
    B, C, H, W = intensities.shape
    _need(intensities, torch.float32, (B, C, H, W), "intensities")
    dev = intensities.device
    wave = _out(wave, (B, T, C, H, W), torch.uint8, dev, "wave")
    t_first = _out(t_first, (B, C, H, W), torch.uint8, dev, "t_first")
    n = spk_rank_latency_workspace_size(B, C, H, W, T)
    ws = _ws(workspace, n, dev)
    _check(_lib.spk_rank_latency(_ptr(intensities), B, C, H, W, T, _ptr(wave), _ptr(t_first), _ptr(ws), n,
                                 _stream(stream)))
    return (wave if wave is not False else None), (t_first if t_first is not False else None)


def spk_local_normalization(intensities, radius, eps=1e-12, out=None, stream=None):
    """Intensities f32 [B,C,H,W] divided by their per-channel regional mean plus eps."""
    B, C, H, W = intensities.shape
    _need(intensities, torch.float32, (B, C, H, W), "intensities")
    out = _out(out, (B, C, H, W), torch.float32, intensities.device, "out")
    _check(_lib.spk_local_normalization(_ptr(intensities), B, C, H, W, radius, float(eps), _ptr(out),
                                        _stream(stream)))
    return out


def spk_expand_wave(t_first, T, wave=None, stream=None):
    """Eq.1: first-spike times u8 [B,C,H,W] -> wave u8 [B,T,C,H,W]."""
    B, C, H, W = t_first.shape
    _need(t_first, torch.uint8, (B, C, H, W), "t_first")
    wave = _out(wave, (B, T, C, H, W), torch.uint8, t_first.device, "wave")
    _check(_lib.spk_expand_wave(_ptr(t_first), B, T, C, H, W, _ptr(wave), _stream(stream)))
    return wave


def spk_validate_wave(wave, bad_count=None, stream=None):
    """Number of neurons breaking Eq.1's structure (device i32 tensor of shape [1])."""
    B, T, C, H, W = wave.shape
    _need(wave, torch.uint8, (B, T, C, H, W), "wave")
    bad_count = _out(bad_count, (1,), torch.int32, wave.device, "bad_count")
    _check(_lib.spk_validate_wave(_ptr(wave), B, T, C, H, W, _ptr(bad_count), _stream(stream)))
    return bad_count


# ---------------------------------------------------------------- conv + fire
def conv_out_size(n, K, pad, stride=1):
    """Eq.2 on the zero-padded input: floor((n + 2 pad - K) / stride) + 1."""
    return (n + 2 * pad - K) // stride + 1


def spk_conv_fire_workspace_size(B, T, Cin, H, W, Cout, K, pad) -> int:
    return int(_lib.spk_conv_fire_workspace_size(B, T, Cin, H, W, Cout, K, pad))


def spk_conv_fire_strided_workspace_size(B, T, Cin, H, W, Cout, K, stride, pad) -> int:
    return int(_lib.spk_conv_fire_strided_workspace_size(B, T, Cin, H, W, Cout, K, stride, pad))


def _conv_call(x, times, T, weight, stride, pad, threshold, potentials, spikes, t_first, v_first, workspace,
               stream):
    """Marshal one conv call; x is the wave u8 [B,T,Cin,H,W] or (times) the
    first-spike map u8 [B,Cin,H,W].  stride None calls the stride-1 entry points."""
    if times:
        B, Cin, H, W = x.shape
        _need(x, torch.uint8, (B, Cin, H, W), "in_t_first")
    else:
        B, T, Cin, H, W = x.shape
        _need(x, torch.uint8, (B, T, Cin, H, W), "wave")
    Cout, Cin2, K, _ = weight.shape
    _need(weight, torch.float32, (Cout, Cin, K, K), "weight")
    s = 1 if stride in (None, "f32") else stride
    Ho, Wo = conv_out_size(H, K, pad, s), conv_out_size(W, K, pad, s)
    dev = x.device
    potentials = _out(potentials, (B, T, Cout, Ho, Wo), torch.float32, dev, "potentials")
    spikes = _out(spikes, (B, T, Cout, Ho, Wo), torch.uint8, dev, "spikes")
    t_first = _out(t_first, (B, Cout, Ho, Wo), torch.uint8, dev, "t_first")
    v_first = _out(v_first, (B, Cout, Ho, Wo), torch.float32, dev, "v_first")
    outs = (_ptr(potentials), _ptr(spikes), _ptr(t_first), _ptr(v_first))
    if stride == "f32":
        n = spk_conv_fire_workspace_size(B, T, Cin, H, W, Cout, K, pad)
        ws = _ws(workspace, n, dev)
        _check(_lib.spk_conv_fire_first_spike_f32mfma(_ptr(x), B, T, Cin, H, W, _ptr(weight), Cout, K, pad,
                                                      float(threshold), *outs, _ptr(ws), n, _stream(stream)))
    elif stride is None:
        n = spk_conv_fire_workspace_size(B, T, Cin, H, W, Cout, K, pad)
        ws = _ws(workspace, n, dev)
        fn = _lib.spk_conv_fire_first_spike if times else _lib.spk_conv_fire
        _check(fn(_ptr(x), B, T, Cin, H, W, _ptr(weight), Cout, K, pad, float(threshold), *outs, _ptr(ws), n,
                  _stream(stream)))
    else:
        n = spk_conv_fire_strided_workspace_size(B, T, Cin, H, W, Cout, K, stride, pad)
        ws = _ws(workspace, n, dev)
        fn = _lib.spk_conv_fire_first_spike_strided if times else _lib.spk_conv_fire_strided
        _check(fn(_ptr(x), B, T, Cin, H, W, _ptr(weight), Cout, K, stride, pad, float(threshold), *outs, _ptr(ws),
                  n, _stream(stream)))
    return potentials, spikes, t_first, v_first


def spk_conv_fire(wave, weight, pad, threshold, potentials=None, spikes=None, t_first=None, v_first=None,
                  workspace=None, stream=None):
    """wave u8 [B,T,Cin,H,W], weight f32 [Cout,Cin,K,K] ->
    (potentials f32 [B,T,Cout,Ho,Wo], spikes u8 [B,T,Cout,Ho,Wo], t_first u8 [B,Cout,Ho,Wo], v_first f32)."""
    return _conv_call(wave, False, None, weight, None, pad, threshold, potentials, spikes, t_first, v_first,
                      workspace, stream)


def spk_conv_fire_first_spike(in_t_first, T, weight, pad, threshold, potentials=None, spikes=None, t_first=None,
                              v_first=None, workspace=None, stream=None):
    """As spk_conv_fire, with the input given by its first-spike map in_t_first u8 [B,Cin,H,W]
    (T = never; the wave it stands for is Eq.1 of it)."""
    return _conv_call(in_t_first, True, T, weight, None, pad, threshold, potentials, spikes, t_first, v_first,
                      workspace, stream)


def spk_conv_fire_pool(in_t_first, T, weight, pad, threshold, pool, potentials=False, spikes=False, t_first=None,
                       v_first=None, pooled_t_first=None, pooled_wave=None, workspace=None, stream=None):
    """Conv + fire + first-spike pooling (window = stride = pool) in one launch:
    -> (potentials or None, spikes or None, t_first, v_first, pooled_t_first u8 [B,Cout,Ho/pool,Wo/pool],
    pooled_wave u8 [B,T,Cout,Ho/pool,Wo/pool] or None).  Per-step outputs default to skipped (False)."""
    B, Cin, H, W = in_t_first.shape
    Cout, Cin2, K, _ = weight.shape
    _need(in_t_first, torch.uint8, (B, Cin, H, W), "in_t_first")
    _need(weight, torch.float32, (Cout, Cin, K, K), "weight")
    Ho, Wo = conv_out_size(H, K, pad), conv_out_size(W, K, pad)
    Hp, Wp = Ho // pool, Wo // pool
    dev = in_t_first.device
    potentials = _out(potentials, (B, T, Cout, Ho, Wo), torch.float32, dev, "potentials")
    spikes = _out(spikes, (B, T, Cout, Ho, Wo), torch.uint8, dev, "spikes")
    t_first = _out(t_first, (B, Cout, Ho, Wo), torch.uint8, dev, "t_first")
    v_first = _out(v_first, (B, Cout, Ho, Wo), torch.float32, dev, "v_first")
    pooled_t_first = _out(pooled_t_first, (B, Cout, Hp, Wp), torch.uint8, dev, "pooled_t_first")
    pooled_wave = _out(pooled_wave, (B, T, Cout, Hp, Wp), torch.uint8, dev, "pooled_wave")
    n = spk_conv_fire_workspace_size(B, T, Cin, H, W, Cout, K, pad)
    ws = _ws(workspace, n, dev)
    _check(_lib.spk_conv_fire_pool(_ptr(in_t_first), B, T, Cin, H, W, _ptr(weight), Cout, K, pad, float(threshold),
                                   int(pool), _ptr(potentials), _ptr(spikes), _ptr(t_first), _ptr(v_first),
                                   _ptr(pooled_t_first), _ptr(pooled_wave), _ptr(ws), n, _stream(stream)))
    none = lambda x: None if x is False else x  # noqa: E731
    return none(potentials), none(spikes), t_first, v_first, pooled_t_first, none(pooled_wave)


def spk_conv_fire_first_spike_f32mfma(in_t_first, T, weight, pad, threshold, potentials=None, spikes=None,
                                      t_first=None, v_first=None, workspace=None, stream=None):
    """spk_conv_fire_first_spike with the contraction on fp32 matrix cores (one fp32 term per weight)."""
    return _conv_call(in_t_first, True, T, weight, "f32", pad, threshold, potentials, spikes, t_first, v_first,
                      workspace, stream)


def spk_conv_fire_strided(wave, weight, stride, pad, threshold, potentials=None, spikes=None, t_first=None,
                          v_first=None, workspace=None, stream=None):
    """spk_conv_fire with stride: output (y, x) reads the padded window at (y*stride, x*stride)."""
    return _conv_call(wave, False, None, weight, int(stride), pad, threshold, potentials, spikes, t_first, v_first,
                      workspace, stream)


def spk_conv_fire_first_spike_strided(in_t_first, T, weight, stride, pad, threshold, potentials=None, spikes=None,
                                      t_first=None, v_first=None, workspace=None, stream=None):
    """spk_conv_fire_first_spike with stride."""
    return _conv_call(in_t_first, True, T, weight, int(stride), pad, threshold, potentials, spikes, t_first, v_first,
                      workspace, stream)


def spk_conv_fire_first_spike_noalloc(in_t_first, T, weight, pad, threshold, potentials=None, spikes=None,
                                      t_first=None, v_first=None, stream=None):
    """As spk_conv_fire_first_spike, with the library's static device scratch
    instead of a workspace (the C call allocates nothing; calls on one GPU must
    not overlap)."""
    B, Cin, H, W = in_t_first.shape
    Cout, Cin2, K, _ = weight.shape
    _need(in_t_first, torch.uint8, (B, Cin, H, W), "in_t_first")
    _need(weight, torch.float32, (Cout, Cin, K, K), "weight")
    Ho, Wo = conv_out_size(H, K, pad), conv_out_size(W, K, pad)
    dev = in_t_first.device
    potentials = _out(potentials, (B, T, Cout, Ho, Wo), torch.float32, dev, "potentials")
    spikes = _out(spikes, (B, T, Cout, Ho, Wo), torch.uint8, dev, "spikes")
    t_first = _out(t_first, (B, Cout, Ho, Wo), torch.uint8, dev, "t_first")
    v_first = _out(v_first, (B, Cout, Ho, Wo), torch.float32, dev, "v_first")
    _check(_lib.spk_conv_fire_first_spike_noalloc(_ptr(in_t_first), B, T, Cin, H, W, _ptr(weight), Cout, K, pad,
                                                  float(threshold), _ptr(potentials), _ptr(spikes), _ptr(t_first),
                                                  _ptr(v_first), _stream(stream)))
    return potentials, spikes, t_first, v_first


# ---------------------------------------------------------------- pool
def pool_out_size(n, kernel, stride, pad):
    return (n + 2 * pad - kernel) // stride + 1


def spk_pool(wave, kernel, stride=None, pad=0, out_wave=None, out_t_first=False, stream=None):
    """Spike max-pooling of wave u8 [B,T,C,H,W] -> (out_wave, out_t_first)."""
    stride = kernel if stride is None else stride
    B, T, C, H, W = wave.shape
    _need(wave, torch.uint8, (B, T, C, H, W), "wave")
    Ho, Wo = pool_out_size(H, kernel, stride, pad), pool_out_size(W, kernel, stride, pad)
    out_wave = _out(out_wave, (B, T, C, Ho, Wo), torch.uint8, wave.device, "out_wave")
    out_t_first = _out(out_t_first, (B, C, Ho, Wo), torch.uint8, wave.device, "out_t_first")
    _check(_lib.spk_pool(_ptr(wave), B, T, C, H, W, kernel, stride, pad, _ptr(out_wave), _ptr(out_t_first),
                         _stream(stream)))
    return out_wave, out_t_first


def spk_pool_first_spike(t_first, T, kernel, stride=None, pad=0, out_wave=None, out_t_first=None, stream=None):
    """Pooling of first-spike times u8 [B,C,H,W] -> (out_wave u8 [B,T,C,Ho,Wo], out_t_first u8 [B,C,Ho,Wo])."""
    stride = kernel if stride is None else stride
    B, C, H, W = t_first.shape
    _need(t_first, torch.uint8, (B, C, H, W), "t_first")
    Ho, Wo = pool_out_size(H, kernel, stride, pad), pool_out_size(W, kernel, stride, pad)
    out_wave = _out(out_wave, (B, T, C, Ho, Wo), torch.uint8, t_first.device, "out_wave")
    out_t_first = _out(out_t_first, (B, C, Ho, Wo), torch.uint8, t_first.device, "out_t_first")
    _check(_lib.spk_pool_first_spike(_ptr(t_first), B, T, C, H, W, kernel, stride, pad, _ptr(out_wave),
                                     _ptr(out_t_first), _stream(stream)))
    return out_wave, out_t_first


def spk_pool_potentials(potentials, kernel, stride=None, pad=0, out=None, stream=None):
    """Max-pooling of potentials f32 [B,T,C,H,W] -> f32 [B,T,C,Ho,Wo] (zero padding)."""
    stride = kernel if stride is None else stride
    B, T, C, H, W = potentials.shape
    _need(potentials, torch.float32, (B, T, C, H, W), "potentials")
    Ho, Wo = pool_out_size(H, kernel, stride, pad), pool_out_size(W, kernel, stride, pad)
    out = _out(out, (B, T, C, Ho, Wo), torch.float32, potentials.device, "out")
    _check(_lib.spk_pool_potentials(_ptr(potentials), B, T, C, H, W, kernel, stride, pad, _ptr(out), _stream(stream)))
    return out


def spk_pointwise_inhibition(t_first, v_first, T, out_t_first=None, out_v_first=None, out_wave=False,
                             potentials=None, stream=None):
    """Per location only the most salient feature keeps its spike: (t_first u8, v_first f32)
    [B,C,H,W] -> (out_t_first, out_v_first, out_wave u8 [B,T,C,H,W] or None); potentials
    f32 [B,T,C,H,W], if given, are masked in place.  out_wave=None allocates the wave."""
    B, C, H, W = t_first.shape
    _need(t_first, torch.uint8, (B, C, H, W), "t_first")
    _need(v_first, torch.float32, (B, C, H, W), "v_first")
    dev = t_first.device
    out_t_first = _out(out_t_first, (B, C, H, W), torch.uint8, dev, "out_t_first")
    out_v_first = _out(out_v_first, (B, C, H, W), torch.float32, dev, "out_v_first")
    out_wave = _out(out_wave, (B, T, C, H, W), torch.uint8, dev, "out_wave")
    if potentials is not None:
        _need(potentials, torch.float32, (B, T, C, H, W), "potentials")
    _check(_lib.spk_pointwise_inhibition(_ptr(t_first), _ptr(v_first), B, T, C, H, W, _ptr(out_t_first),
                                         _ptr(out_v_first), _ptr(out_wave), _ptr(potentials), _stream(stream)))
    return out_t_first, out_v_first, (out_wave if out_wave is not False else None)


# ---------------------------------------------------------------- kWTA
def spk_kwta_workspace_size(B, C, H, W) -> int:
    return int(_lib.spk_kwta_workspace_size(B, C, H, W))


def spk_kwta(t_first, v_first, T, k, radius, winners=None, n_winners=None, workspace=None, stream=None):
    """(t_first u8, v_first f32) [B,C,H,W] -> (winners i32 [B,k,4] = (f,t,y,x), n_winners i32 [B])."""
    B, C, H, W = t_first.shape
    _need(t_first, torch.uint8, (B, C, H, W), "t_first")
    _need(v_first, torch.float32, (B, C, H, W), "v_first")
    dev = t_first.device
    winners = _out(winners, (B, k, 4), torch.int32, dev, "winners")
    n_winners = _out(n_winners, (B,), torch.int32, dev, "n_winners")
    n = spk_kwta_workspace_size(B, C, H, W)
    ws = _ws(workspace, n, dev)
    _check(_lib.spk_kwta(_ptr(t_first), _ptr(v_first), B, T, C, H, W, k, radius, _ptr(winners), _ptr(n_winners),
                         _ptr(ws), n, _stream(stream)))
    return winners, n_winners


# ---------------------------------------------------------------- plasticity
def _stdp_args(weight, pre_wave, winners, n_winners, T=None):
    """Sizes of a plasticity call; with T given, pre_wave is the first-spike map [B,Cin,H,W]."""
    Cout, Cin, K, _ = weight.shape
    if T is None:
        B, T, Cin2, H, W = pre_wave.shape
        _need(pre_wave, torch.uint8, (B, T, Cin, H, W), "pre_wave")
    else:
        B, Cin2, H, W = pre_wave.shape
        _need(pre_wave, torch.uint8, (B, Cin, H, W), "pre_t_first")
    k = winners.shape[1]
    _need(weight, torch.float32, (Cout, Cin, K, K), "weight")
    _need(winners, torch.int32, (B, k, 4), "winners")
    _need(n_winners, torch.int32, (B,), "n_winners")
    return Cout, Cin, K, B, T, H, W, k


def spk_stdp_workspace_size(Cout, Cin, K, B, k) -> int:
    return int(_lib.spk_stdp_workspace_size(Cout, Cin, K, B, k))


def _stdp_call(weight, stride, pad, pre_wave, winners, n_winners, reward, a_plus, a_minus, lb, ub, stabilizer,
               workspace, stream, T=None):
    Cout, Cin, K, B, T, H, W, k = _stdp_args(weight, pre_wave, winners, n_winners, T)
    if reward is not None:
        _need(reward, torch.int8, (B,), "reward")
    n = spk_stdp_workspace_size(Cout, Cin, K, B, k)
    ws = _ws(workspace, n, weight.device)
    mid = (_ptr(pre_wave), B, T, H, W, _ptr(winners), _ptr(n_winners), k) + (() if reward is None else (_ptr(reward),))
    tail = (float(a_plus), float(a_minus), float(lb), float(ub), int(bool(stabilizer)), _ptr(ws), n, _stream(stream))
    if stride == "times":  # first-spike map input (stride 1)
        head = (_ptr(weight), Cout, Cin, K, pad)
        fn = _lib.spk_rstdp_first_spike if reward is not None else _lib.spk_stdp_first_spike
    else:
        head = (_ptr(weight), Cout, Cin, K) + ((pad,) if stride is None else (stride, pad))
        fn = {(False, False): _lib.spk_stdp, (True, False): _lib.spk_rstdp, (False, True): _lib.spk_stdp_strided,
              (True, True): _lib.spk_rstdp_strided}[(reward is not None, stride is not None)]
    _check(fn(*head, *mid, *tail))
    return weight


def spk_stdp(weight, pad, pre_wave, winners, n_winners, a_plus, a_minus, lb=0.0, ub=1.0, stabilizer=True,
             workspace=None, stream=None):
    """Eq.4 on the winners' weights (in place on `weight`), ordered replay over images."""
    return _stdp_call(weight, None, pad, pre_wave, winners, n_winners, None, a_plus, a_minus, lb, ub, stabilizer,
                      workspace, stream)


def spk_rstdp(weight, pad, pre_wave, winners, n_winners, reward, a_plus, a_minus, lb=0.0, ub=1.0, stabilizer=True,
              workspace=None, stream=None):
    """R-STDP: reward i8 [B] in {+1,-1,0} selects STDP, anti-STDP or nothing per image."""
    return _stdp_call(weight, None, pad, pre_wave, winners, n_winners, reward, a_plus, a_minus, lb, ub, stabilizer,
                      workspace, stream)


def spk_stdp_first_spike(weight, pad, pre_t_first, T, winners, n_winners, a_plus, a_minus, lb=0.0, ub=1.0,
                         stabilizer=True, workspace=None, stream=None):
    """spk_stdp with the layer input given by its first-spike map u8 [B,Cin,H,W] (T = never)."""
    return _stdp_call(weight, "times", pad, pre_t_first, winners, n_winners, None, a_plus, a_minus, lb, ub,
                      stabilizer, workspace, stream, T=T)


def spk_rstdp_first_spike(weight, pad, pre_t_first, T, winners, n_winners, reward, a_plus, a_minus, lb=0.0, ub=1.0,
                          stabilizer=True, workspace=None, stream=None):
    """spk_rstdp with the layer input given by its first-spike map."""
    return _stdp_call(weight, "times", pad, pre_t_first, winners, n_winners, reward, a_plus, a_minus, lb, ub,
                      stabilizer, workspace, stream, T=T)


def spk_stdp_strided(weight, stride, pad, pre_wave, winners, n_winners, a_plus, a_minus, lb=0.0, ub=1.0,
                     stabilizer=True, workspace=None, stream=None):
    """spk_stdp of a layer with stride (winner (y, x) sees the input window at (y*stride, x*stride))."""
    return _stdp_call(weight, int(stride), pad, pre_wave, winners, n_winners, None, a_plus, a_minus, lb, ub,
                      stabilizer, workspace, stream)


def spk_rstdp_strided(weight, stride, pad, pre_wave, winners, n_winners, reward, a_plus, a_minus, lb=0.0, ub=1.0,
                      stabilizer=True, workspace=None, stream=None):
    """spk_rstdp of a layer with stride."""
    return _stdp_call(weight, int(stride), pad, pre_wave, winners, n_winners, reward, a_plus, a_minus, lb, ub,
                      stabilizer, workspace, stream)


def spk_decide(winners, n_winners, labels, n_classes=10, decision=None, reward=None, stream=None):
    """(decision i32 [B], reward i8 [B]) from the first winner's feature mod n_classes."""
    B, k, _ = winners.shape
    _need(winners, torch.int32, (B, k, 4), "winners")
    _need(n_winners, torch.int32, (B,), "n_winners")
    _need(labels, torch.int32, (B,), "labels")
    decision = _out(decision, (B,), torch.int32, winners.device, "decision")
    reward = _out(reward, (B,), torch.int8, winners.device, "reward")
    _check(_lib.spk_decide(_ptr(winners), _ptr(n_winners), B, k, _ptr(labels), n_classes, _ptr(decision),
                           _ptr(reward), _stream(stream)))
    return decision, reward


def spk_count_events(wave, Cout, K, pad, count=None, stream=None):
    """Synaptic events (spiking pre, post pairs) of a conv over wave u8 [B,T,Cin,H,W] -> device int64 [1]."""
    B, T, Cin, H, W = wave.shape
    _need(wave, torch.uint8, (B, T, Cin, H, W), "wave")
    count = _out(count, (1,), torch.int64, wave.device, "count")
    _check(_lib.spk_count_events(_ptr(wave), B, T, Cin, H, W, Cout, K, pad, _ptr(count), _stream(stream)))
    return count


def spk_count_events_strided(wave, Cout, K, stride, pad, count=None, stream=None):
    """spk_count_events of a conv with stride."""
    B, T, Cin, H, W = wave.shape
    _need(wave, torch.uint8, (B, T, Cin, H, W), "wave")
    count = _out(count, (1,), torch.int64, wave.device, "count")
    _check(_lib.spk_count_events_strided(_ptr(wave), B, T, Cin, H, W, Cout, K, int(stride), pad, _ptr(count),
                                         _stream(stream)))
    return count


INF = math.inf
