"""Python binding of libquartz.so (the QuaRTZ W4A4 linear hot path on gfx950).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch is used for device memory and the current stream.  The
functions named like the C entry points (``quartz_quantize_act`` ...) take raw
integers (device addresses, sizes) and return the status code; the tensor
helpers (``quantize_act``, ``pack_weight``, ``w4a4_linear`` ...) allocate the
outputs with ``torch.empty`` on the input's device and raise ``QuartzError`` on
a non-OK status.  There is no fallback: if ``libquartz.so`` is missing or fails
to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

__all__ = [
    "QuartzError", "library_path", "load",
    "quartz_quantize_act", "quartz_packed_weight_bytes", "quartz_pack_weight",
    "quartz_w4a4_linear", "quartz_w4a4_linear_workspace_bytes", "quartz_w4a4_linear_ws",
    "quartz_w4a4_linear_schedule", "quartz_unpack_weight", "quartz_w4a4_gemm_i32",
    "quartz_w4a4_linear_quantize", "quartz_quantize_act_static", "quartz_pack_weight_per_channel",
    "quartz_w4a4_linear_static", "quartz_weight_group_sums", "quartz_w4a4_linear_asym",
    "quartz_w4a4_conv3x3", "quartz_w4a4_conv3x3_static",
    "quartz_w4a4_linear_noalloc", "quartz_w4a4_linear_noalloc_max_bytes", "w4a4_linear_noalloc",
    "quartz_status_string", "QuantizedAct", "PackedWeight",
    "quantize_act", "pack_weight", "w4a4_linear", "w4a4_linear_quantize", "gemm_workspace",
    "quantize_act_static", "pack_weight_per_channel", "w4a4_linear_static", "weight_group_sums",
    "w4a4_linear_asym", "linear_schedule", "w4a4_conv3x3", "w4a4_conv3x3_static",
    "unpack_weight", "w4a4_gemm_i32", "EXPORTED_SYMBOLS",
    "MODE_SYMMETRIC", "MODE_ASYMMETRIC", "MODE_STATIC",
    "quartz_quantize_vt", "quartz_attn_scores", "quartz_softmax_quantize",
    "quartz_attn_pv_workspace_bytes", "quartz_attn_pv", "quartz_lzs_attention_workspace_bytes",
    "quartz_lzs_attention", "quantize_vt", "attn_scores", "softmax_quantize", "attn_pv",
    "attention_workspace", "lzs_attention",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libquartz.so")

QUARTZ_OK = 0
MODE_SYMMETRIC = 0
MODE_ASYMMETRIC = 1
# binding-side tag of activations from quantize_act_static (no per-group scales)
MODE_STATIC = 2
EPI_NONE = 0
EPI_GELU_TANH = 1
GROUP = 64

EXPORTED_SYMBOLS = (
    "quartz_quantize_act", "quartz_packed_weight_bytes", "quartz_pack_weight",
    "quartz_w4a4_linear", "quartz_w4a4_linear_workspace_bytes", "quartz_w4a4_linear_ws",
    "quartz_w4a4_linear_schedule", "quartz_unpack_weight", "quartz_w4a4_gemm_i32",
    "quartz_w4a4_linear_quantize", "quartz_quantize_act_static", "quartz_pack_weight_per_channel",
    "quartz_w4a4_linear_static", "quartz_weight_group_sums", "quartz_w4a4_linear_asym",
    "quartz_w4a4_conv3x3", "quartz_w4a4_conv3x3_static", "quartz_status_string",
    "quartz_w4a4_linear_noalloc", "quartz_w4a4_linear_noalloc_max_bytes",
    "quartz_quantize_vt", "quartz_attn_scores", "quartz_softmax_quantize",
    "quartz_attn_pv_workspace_bytes", "quartz_attn_pv", "quartz_lzs_attention_workspace_bytes",
    "quartz_lzs_attention",
)


class QuartzError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {quartz_status_string(status)} (status {status})")


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load libquartz.so (built in-tree by build.py); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"libquartz.so not found at {_LIB_PATH}; build it with "
            "`python paper_2509_26436_amd/build.py` (no CPU fallback exists)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.quartz_quantize_act.argtypes = [P, I64, I64, I64, I32, I32, I32, P, P, P, P, P]
    lib.quartz_quantize_act.restype = I32
    lib.quartz_packed_weight_bytes.argtypes = [I64, I64, I32]
    lib.quartz_packed_weight_bytes.restype = SZ
    lib.quartz_pack_weight.argtypes = [P, I64, I64, I32, P, P, P]
    lib.quartz_pack_weight.restype = I32
    lib.quartz_w4a4_linear.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I32, I32, I32, P]
    lib.quartz_w4a4_linear.restype = I32
    lib.quartz_w4a4_linear_workspace_bytes.argtypes = [I64, I64, I64, I32]
    lib.quartz_w4a4_linear_workspace_bytes.restype = SZ
    lib.quartz_w4a4_linear_ws.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I32, I32, I32,
                                          P, SZ, P]
    lib.quartz_w4a4_linear_ws.restype = I32
    lib.quartz_w4a4_linear_noalloc.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I32, I32,
                                               I32, P]
    lib.quartz_w4a4_linear_noalloc.restype = I32
    lib.quartz_w4a4_linear_noalloc_max_bytes.argtypes = []
    lib.quartz_w4a4_linear_noalloc_max_bytes.restype = SZ
    F32 = ctypes.c_float
    lib.quartz_quantize_act_static.argtypes = [P, I64, I64, I64, F32, I32, P, P, P]
    lib.quartz_quantize_act_static.restype = I32
    lib.quartz_pack_weight_per_channel.argtypes = [P, I64, I64, P, P, P]
    lib.quartz_pack_weight_per_channel.restype = I32
    lib.quartz_w4a4_linear_static.argtypes = [P, P, F32, P, P, P, I64, I64, I64, I64, I32, I32, P,
                                              ctypes.c_size_t, P]
    lib.quartz_w4a4_linear_static.restype = I32
    lib.quartz_weight_group_sums.argtypes = [P, I64, I64, I32, P, P]
    lib.quartz_weight_group_sums.restype = I32
    lib.quartz_w4a4_linear_asym.argtypes = [P, P, P, P, P, P, P, P, I64, I64, I64, I64, I32, I32,
                                            I32, P, ctypes.c_size_t, P]
    lib.quartz_w4a4_linear_asym.restype = I32
    lib.quartz_w4a4_linear_quantize.argtypes = [P, P, P, P, P, P, I64, I64, I64, I32, I32, I32,
                                                I32, I32, P, P, P, P, P, ctypes.c_size_t, P]
    lib.quartz_w4a4_linear_quantize.restype = I32
    lib.quartz_w4a4_conv3x3.argtypes = [P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I32, I32,
                                        I32, P, SZ, P]
    lib.quartz_w4a4_conv3x3.restype = I32
    lib.quartz_w4a4_conv3x3_static.argtypes = [P, P, F32, P, P, P, I64, I64, I64, I64, I64, I64,
                                               I32, I32, P, SZ, P]
    lib.quartz_w4a4_conv3x3_static.restype = I32
    lib.quartz_w4a4_linear_schedule.argtypes = [I64, I64, I64, I32, I32, I32, P, P, I64]
    lib.quartz_w4a4_linear_schedule.restype = I64
    lib.quartz_unpack_weight.argtypes = [P, I64, I64, I32, P, P]
    lib.quartz_unpack_weight.restype = I32
    lib.quartz_w4a4_gemm_i32.argtypes = [P, P, P, P, I64, I64, I64, I32, I32, P]
    lib.quartz_w4a4_gemm_i32.restype = I32
    lib.quartz_quantize_vt.argtypes = [P, I64, I64, I64, I64, I32, P, P, P, P]
    lib.quartz_quantize_vt.restype = I32
    lib.quartz_attn_scores.argtypes = [P, P, P, I64, I64, P, P, P, I64, I64, I64, I64, I64, I32,
                                       F32, P, I64, P]
    lib.quartz_attn_scores.restype = I32
    lib.quartz_softmax_quantize.argtypes = [P, I64, I64, I64, I32, P, P, P, P]
    lib.quartz_softmax_quantize.restype = I32
    lib.quartz_attn_pv_workspace_bytes.argtypes = [I64, I64, I64]
    lib.quartz_attn_pv_workspace_bytes.restype = SZ
    lib.quartz_attn_pv.argtypes = [P, P, P, P, P, P, I64, I64, I64, I64, I64, I32, P, I64, P, SZ,
                                   P]
    lib.quartz_attn_pv.restype = I32
    lib.quartz_lzs_attention_workspace_bytes.argtypes = [I64, I64, I64, I32]
    lib.quartz_lzs_attention_workspace_bytes.restype = SZ
    lib.quartz_lzs_attention.argtypes = [P, P, P, I64, I64, I64, I32, P, I64, P, SZ, P]
    lib.quartz_lzs_attention.restype = I32
    lib.quartz_status_string.argtypes = [I32]
    lib.quartz_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


# ----------------------------------------------------------- raw C entry points

def quartz_status_string(status: int) -> str:
    return load().quartz_status_string(int(status)).decode()


def quartz_quantize_act(x, M, K, ldx, group_size, lzs_group, mode, codes, flags, scales,
                        zeros, stream) -> int:
    return load().quartz_quantize_act(x, M, K, ldx, group_size, lzs_group, mode, codes, flags,
                                      scales, zeros, stream)


def quartz_packed_weight_bytes(N, K, group_size=GROUP) -> int:
    return int(load().quartz_packed_weight_bytes(N, K, group_size))


def quartz_pack_weight(w, N, K, group_size, w_packed, w_scales, stream) -> int:
    return load().quartz_pack_weight(w, N, K, group_size, w_packed, w_scales, stream)


def quartz_w4a4_linear(codes, flags, scales, zeros, w_packed, bias, y, M, N, K, ldy,
                       group_size, lzs_group, epilogue, stream) -> int:
    return load().quartz_w4a4_linear(codes, flags, scales, zeros, w_packed, bias, y, M, N, K, ldy,
                                     group_size, lzs_group, epilogue, stream)


def quartz_w4a4_linear_workspace_bytes(M, N, K, group_size=GROUP) -> int:
    return int(load().quartz_w4a4_linear_workspace_bytes(M, N, K, group_size))


def quartz_w4a4_linear_ws(codes, flags, scales, zeros, w_packed, bias, y, M, N, K, ldy,
                          group_size, lzs_group, epilogue, workspace, workspace_bytes,
                          stream) -> int:
    return load().quartz_w4a4_linear_ws(codes, flags, scales, zeros, w_packed, bias, y, M, N, K,
                                        ldy, group_size, lzs_group, epilogue, workspace,
                                        workspace_bytes, stream)


def quartz_w4a4_linear_noalloc(codes, flags, scales, zeros, w_packed, bias, y, M, N, K, ldy,
                               group_size, lzs_group, epilogue, stream) -> int:
    return load().quartz_w4a4_linear_noalloc(codes, flags, scales, zeros, w_packed, bias, y, M, N,
                                             K, ldy, group_size, lzs_group, epilogue, stream)


def quartz_w4a4_linear_noalloc_max_bytes() -> int:
    return int(load().quartz_w4a4_linear_noalloc_max_bytes())


def quartz_w4a4_linear_quantize(codes, flags, scales, zeros, w_packed, bias, M, N, K,
                                group_size, lzs_group, epilogue, out_lzs_group, out_mode,
                                out_codes, out_flags, out_scales, out_zeros, workspace,
                                workspace_bytes, stream) -> int:
    return load().quartz_w4a4_linear_quantize(codes, flags, scales, zeros, w_packed, bias, M, N,
                                              K, group_size, lzs_group, epilogue, out_lzs_group,
                                              out_mode, out_codes, out_flags, out_scales,
                                              out_zeros, workspace, workspace_bytes, stream)


def quartz_quantize_act_static(x, M, K, ldx, scale, lzs_group, codes, flags, stream) -> int:
    return load().quartz_quantize_act_static(x, M, K, ldx, scale, lzs_group, codes, flags, stream)


def quartz_pack_weight_per_channel(w, N, K, w_packed, w_scales, stream) -> int:
    return load().quartz_pack_weight_per_channel(w, N, K, w_packed, w_scales, stream)


def quartz_w4a4_linear_static(codes, flags, act_scale, w_packed, bias, y, M, N, K, ldy,
                              lzs_group, epilogue, workspace, workspace_bytes, stream) -> int:
    return load().quartz_w4a4_linear_static(codes, flags, act_scale, w_packed, bias, y, M, N, K,
                                            ldy, lzs_group, epilogue, workspace, workspace_bytes,
                                            stream)


def quartz_weight_group_sums(w_packed, N, K, group_size, w_sums, stream) -> int:
    return load().quartz_weight_group_sums(w_packed, N, K, group_size, w_sums, stream)


def quartz_w4a4_linear_asym(codes, flags, scales, zeros, w_packed, w_sums, bias, y, M, N, K,
                            ldy, group_size, lzs_group, epilogue, workspace, workspace_bytes,
                            stream) -> int:
    return load().quartz_w4a4_linear_asym(codes, flags, scales, zeros, w_packed, w_sums, bias, y,
                                          M, N, K, ldy, group_size, lzs_group, epilogue,
                                          workspace, workspace_bytes, stream)


def quartz_w4a4_conv3x3(codes, flags, scales, w_packed, bias, y, images, H, W, C, N, ldy,
                        group_size, lzs_group, epilogue, workspace, workspace_bytes, stream) -> int:
    return load().quartz_w4a4_conv3x3(codes, flags, scales, w_packed, bias, y, images, H, W, C, N,
                                      ldy, group_size, lzs_group, epilogue, workspace,
                                      workspace_bytes, stream)


def quartz_w4a4_conv3x3_static(codes, flags, act_scale, w_packed, bias, y, images, H, W, C, N,
                               ldy, lzs_group, epilogue, workspace, workspace_bytes,
                               stream) -> int:
    return load().quartz_w4a4_conv3x3_static(codes, flags, act_scale, w_packed, bias, y, images,
                                             H, W, C, N, ldy, lzs_group, epilogue, workspace,
                                             workspace_bytes, stream)


def quartz_w4a4_linear_schedule(M, N, K, blocks, split, tiles, schedule, segments, capacity) -> int:
    return int(load().quartz_w4a4_linear_schedule(M, N, K, blocks, split, tiles, schedule, segments,
                                                  capacity))


def quartz_unpack_weight(w_packed, N, K, group_size, wq, stream) -> int:
    return load().quartz_unpack_weight(w_packed, N, K, group_size, wq, stream)


def quartz_w4a4_gemm_i32(codes, flags, w_packed, acc, M, N, K, group_size, lzs_group,
                         stream) -> int:
    return load().quartz_w4a4_gemm_i32(codes, flags, w_packed, acc, M, N, K, group_size,
                                       lzs_group, stream)


def quartz_quantize_vt(v, heads, L, d, ldv, lzs_group, codes, flags, scales, stream) -> int:
    return load().quartz_quantize_vt(v, heads, L, d, ldv, lzs_group, codes, flags, scales, stream)


def quartz_attn_scores(qc, qf, qs, q_plane, q_row0, kc, kf, ks, k_plane, k_row0, Lq, Lk, d,
                       lzs_group, scale, s, lds, stream) -> int:
    return load().quartz_attn_scores(qc, qf, qs, q_plane, q_row0, kc, kf, ks, k_plane, k_row0, Lq,
                                     Lk, d, lzs_group, scale, s, lds, stream)


def quartz_softmax_quantize(s, M, N, lds, lzs_group, codes, flags, scales, stream) -> int:
    return load().quartz_softmax_quantize(s, M, N, lds, lzs_group, codes, flags, scales, stream)


def quartz_attn_pv_workspace_bytes(Lq, Lk, d) -> int:
    return int(load().quartz_attn_pv_workspace_bytes(Lq, Lk, d))


def quartz_attn_pv(pc, pf, ps, vc, vf, vs, vt_plane, vt_row0, Lq, Lk, d, lzs_group, o, ldo,
                   workspace, workspace_bytes, stream) -> int:
    return load().quartz_attn_pv(pc, pf, ps, vc, vf, vs, vt_plane, vt_row0, Lq, Lk, d, lzs_group,
                                 o, ldo, workspace, workspace_bytes, stream)


def quartz_lzs_attention_workspace_bytes(heads, L, d, lzs_group) -> int:
    return int(load().quartz_lzs_attention_workspace_bytes(heads, L, d, lzs_group))


def quartz_lzs_attention(q, k, v, heads, L, d, lzs_group, o, ldo, workspace, workspace_bytes,
                         stream) -> int:
    return load().quartz_lzs_attention(q, k, v, heads, L, d, lzs_group, o, ldo, workspace,
                                       workspace_bytes, stream)


# ------------------------------------------------------------- tensor helpers

def _torch():
    import torch
    return torch


def _stream_handle(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(status: int, what: str):
    if status != QUARTZ_OK:
        raise QuartzError(status, what)


@dataclass
class QuantizedAct:
    """Quantizer outputs, K-group-major (see include/quartz.h)."""
    codes: "object"     # uint8 [K/64, M, 32]
    flags: "object"     # uint8 [K/64, M, 64/lzs_group]
    scales: "object"    # int16 [K/64, M] (fp16 bit patterns)
    zeros: "object"     # int8 [K/64, M] or None
    M: int
    K: int
    lzs_group: int
    mode: int = MODE_SYMMETRIC   # MODE_SYMMETRIC, MODE_ASYMMETRIC or MODE_STATIC


_LAYER_FOR_MODE = {MODE_SYMMETRIC: "w4a4_linear / w4a4_linear_quantize / w4a4_conv3x3",
                   MODE_ASYMMETRIC: "w4a4_linear_asym",
                   MODE_STATIC: "w4a4_linear_static / w4a4_conv3x3_static"}


def _need_mode(a: "QuantizedAct", mode: int, what: str):
    """Each layer decodes one quantizer mode: symmetric codes fed to the
    asymmetric layer (or the reverse) would give wrong outputs silently."""
    if a.mode != mode:
        raise ValueError(f"{what} needs activations quantized in mode {mode}, got mode {a.mode}; "
                         f"use {_LAYER_FOR_MODE.get(a.mode, 'the matching layer')}")


@dataclass
class PackedWeight:
    data: "object"      # uint8 [quartz_packed_weight_bytes]
    scales: "object"    # int16 [N, K/64] (fp16 bit patterns) or None
    N: int
    K: int


def quantize_act(x, lzs_group: int = 16, with_zeros: bool = False, stream=None,
                 out: QuantizedAct | None = None, mode: int = MODE_SYMMETRIC) -> QuantizedAct:
    """x: bf16 [M, K] CUDA tensor whose rows are 16-byte aligned (stride(1) == 1).
    ``mode=MODE_ASYMMETRIC`` always returns the zero points."""
    torch = _torch()
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
    M, K = x.shape
    ldx = x.stride(0)
    if out is None:
        dev = x.device
        G = K // GROUP
        out = QuantizedAct(
            codes=torch.empty((G, M, 32), dtype=torch.uint8, device=dev),
            flags=torch.empty((G, M, GROUP // lzs_group), dtype=torch.uint8, device=dev),
            scales=torch.empty((G, M), dtype=torch.int16, device=dev),
            zeros=(torch.empty((G, M), dtype=torch.int8, device=dev)
                   if with_zeros or mode == MODE_ASYMMETRIC else None),
            M=M, K=K, lzs_group=lzs_group, mode=mode)
    else:
        out.mode = mode
    st = quartz_quantize_act(_ptr(x), M, K, ldx, GROUP, lzs_group, mode,
                             _ptr(out.codes), _ptr(out.flags), _ptr(out.scales), _ptr(out.zeros),
                             _stream_handle(stream))
    _check(st, "quartz_quantize_act")
    return out


def pack_weight(w, with_scales: bool = True, stream=None) -> PackedWeight:
    """w: bf16 [N, K] contiguous CUDA tensor (nn.Linear weight layout)."""
    torch = _torch()
    if w.dtype != torch.bfloat16 or w.dim() != 2 or not w.is_contiguous():
        raise ValueError("w must be a contiguous 2-D bf16 tensor")
    N, K = w.shape
    nbytes = quartz_packed_weight_bytes(N, K, GROUP)
    data = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=w.device)
    scales = torch.empty((N, K // GROUP), dtype=torch.int16, device=w.device) if with_scales else None
    st = quartz_pack_weight(_ptr(w), N, K, GROUP, _ptr(data), _ptr(scales), _stream_handle(stream))
    _check(st, "quartz_pack_weight")
    return PackedWeight(data=data, scales=scales, N=N, K=K)


def gemm_workspace(M: int, N: int, K: int, device):
    """Zero-filled uint8 workspace for ``w4a4_linear(..., workspace=...)`` on ``device`` (the
    current device's size query), or None when this shape needs none."""
    torch = _torch()
    nbytes = quartz_w4a4_linear_workspace_bytes(M, N, K, GROUP)
    return torch.zeros((nbytes,), dtype=torch.uint8, device=device) if nbytes else None


def w4a4_linear(a: QuantizedAct, w: PackedWeight, bias=None, epilogue: int = EPI_NONE,
                out=None, stream=None, workspace=None):
    """Returns y bf16 [M, N] (or writes ``out``, a bf16 [M, >=N] view with unit column stride).
    With ``workspace`` (from ``gemm_workspace``) the call is quartz_w4a4_linear_ws."""
    torch = _torch()
    _need_mode(a, MODE_SYMMETRIC, "w4a4_linear")
    if a.K != w.K:
        raise ValueError("K mismatch between activations and weights")
    if bias is not None and (bias.dtype != torch.bfloat16 or bias.numel() != w.N):
        raise ValueError("bias must be bf16 [N]")
    if out is None:
        out = torch.empty((a.M, w.N), dtype=torch.bfloat16, device=a.codes.device)
    ldy = out.stride(0)
    if workspace is None:
        st = quartz_w4a4_linear(_ptr(a.codes), _ptr(a.flags), _ptr(a.scales), _ptr(a.zeros),
                                _ptr(w.data), _ptr(bias), _ptr(out), a.M, w.N, a.K, ldy, GROUP,
                                a.lzs_group, epilogue, _stream_handle(stream))
        _check(st, "quartz_w4a4_linear")
    else:
        st = quartz_w4a4_linear_ws(_ptr(a.codes), _ptr(a.flags), _ptr(a.scales), _ptr(a.zeros),
                                   _ptr(w.data), _ptr(bias), _ptr(out), a.M, w.N, a.K, ldy,
                                   GROUP, a.lzs_group, epilogue, _ptr(workspace),
                                   workspace.numel() * workspace.element_size(),
                                   _stream_handle(stream))
        _check(st, "quartz_w4a4_linear_ws")
    return out


def w4a4_linear_noalloc(a: QuantizedAct, w: PackedWeight, out, bias=None,
                        epilogue: int = EPI_NONE, stream=None):
    """quartz_w4a4_linear_noalloc into the caller's ``out`` (bf16 [M, >=N] with unit
    column stride): the split layer of ``w4a4_linear(..., workspace=...)`` using the
    library's device scratch array, so this call allocates nothing."""
    torch = _torch()
    _need_mode(a, MODE_SYMMETRIC, "w4a4_linear_noalloc")
    if a.K != w.K:
        raise ValueError("K mismatch between activations and weights")
    if bias is not None and (bias.dtype != torch.bfloat16 or bias.numel() != w.N):
        raise ValueError("bias must be bf16 [N]")
    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1 or \
            out.shape[0] != a.M or out.shape[1] < w.N:
        raise ValueError("out must be a bf16 [M, >=N] tensor with unit column stride")
    st = quartz_w4a4_linear_noalloc(_ptr(a.codes), _ptr(a.flags), _ptr(a.scales), _ptr(a.zeros),
                                    _ptr(w.data), _ptr(bias), _ptr(out), a.M, w.N, a.K,
                                    out.stride(0), GROUP, a.lzs_group, epilogue,
                                    _stream_handle(stream))
    _check(st, "quartz_w4a4_linear_noalloc")
    return out


def _empty_act(M: int, K: int, lzs_group: int, with_zeros: bool, device) -> QuantizedAct:
    torch = _torch()
    G = K // GROUP
    return QuantizedAct(
        codes=torch.empty((G, M, 32), dtype=torch.uint8, device=device),
        flags=torch.empty((G, M, GROUP // lzs_group), dtype=torch.uint8, device=device),
        scales=torch.empty((G, M), dtype=torch.int16, device=device),
        zeros=torch.empty((G, M), dtype=torch.int8, device=device) if with_zeros else None,
        M=M, K=K, lzs_group=lzs_group)


def w4a4_linear_quantize(a: QuantizedAct, w: PackedWeight, bias=None, epilogue: int = EPI_NONE,
                         out_lzs_group: int = 16, with_zeros: bool = False,
                         out: QuantizedAct | None = None, stream=None, workspace=None):
    """The layer's output quantized for the next layer (quartz_w4a4_linear_quantize): a
    QuantizedAct with M = a.M rows and K = w.N (w.N % 64 == 0), equal to
    ``quantize_act(w4a4_linear(a, w, ...), out_lzs_group)``."""
    torch = _torch()
    _need_mode(a, MODE_SYMMETRIC, "w4a4_linear_quantize")
    if a.K != w.K:
        raise ValueError("K mismatch between activations and weights")
    if bias is not None and (bias.dtype != torch.bfloat16 or bias.numel() != w.N):
        raise ValueError("bias must be bf16 [N]")
    if out is None:
        out = _empty_act(a.M, w.N, out_lzs_group, with_zeros, a.codes.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = quartz_w4a4_linear_quantize(_ptr(a.codes), _ptr(a.flags), _ptr(a.scales), _ptr(a.zeros),
                                     _ptr(w.data), _ptr(bias), a.M, w.N, a.K, GROUP, a.lzs_group,
                                     epilogue, out.lzs_group, MODE_SYMMETRIC, _ptr(out.codes),
                                     _ptr(out.flags), _ptr(out.scales), _ptr(out.zeros),
                                     _ptr(workspace), nbytes, _stream_handle(stream))
    _check(st, "quartz_w4a4_linear_quantize")
    return out


def quantize_act_static(x, scale: float, lzs_group: int = 16, stream=None,
                        out: QuantizedAct | None = None) -> QuantizedAct:
    """LDM setting: x bf16 [M, K] quantized with one per-tensor fp32 ``scale``
    (quartz_quantize_act_static); the result has no scales or zero points."""
    torch = _torch()
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bf16 tensor with unit column stride")
    M, K = x.shape
    if out is None:
        G = K // GROUP
        out = QuantizedAct(
            codes=torch.empty((G, M, 32), dtype=torch.uint8, device=x.device),
            flags=torch.empty((G, M, GROUP // lzs_group), dtype=torch.uint8, device=x.device),
            scales=None, zeros=None, M=M, K=K, lzs_group=lzs_group, mode=MODE_STATIC)
    else:
        out.mode = MODE_STATIC
    st = quartz_quantize_act_static(_ptr(x), M, K, x.stride(0), float(scale), lzs_group,
                                    _ptr(out.codes), _ptr(out.flags), _stream_handle(stream))
    _check(st, "quartz_quantize_act_static")
    return out


def pack_weight_per_channel(w, with_scales: bool = True, stream=None) -> PackedWeight:
    """LDM setting: w bf16 [N, K] packed with one fp16 scale per output channel
    (``scales``: int16 [N] fp16 bit patterns)."""
    torch = _torch()
    if w.dtype != torch.bfloat16 or w.dim() != 2 or not w.is_contiguous():
        raise ValueError("w must be a contiguous 2-D bf16 tensor")
    N, K = w.shape
    nbytes = quartz_packed_weight_bytes(N, K, GROUP)
    data = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=w.device)
    scales = torch.empty((N,), dtype=torch.int16, device=w.device) if with_scales else None
    st = quartz_pack_weight_per_channel(_ptr(w), N, K, _ptr(data), _ptr(scales),
                                        _stream_handle(stream))
    _check(st, "quartz_pack_weight_per_channel")
    return PackedWeight(data=data, scales=scales, N=N, K=K)


def w4a4_linear_static(a: QuantizedAct, w: PackedWeight, act_scale: float, bias=None,
                       epilogue: int = EPI_NONE, out=None, stream=None, workspace=None):
    """LDM-setting layer (quartz_w4a4_linear_static): ``a`` from quantize_act_static with
    ``act_scale``, ``w`` from pack_weight_per_channel; returns y bf16 [M, N]."""
    torch = _torch()
    _need_mode(a, MODE_STATIC, "w4a4_linear_static")
    if a.K != w.K:
        raise ValueError("K mismatch between activations and weights")
    if bias is not None and (bias.dtype != torch.bfloat16 or bias.numel() != w.N):
        raise ValueError("bias must be bf16 [N]")
    if out is None:
        out = torch.empty((a.M, w.N), dtype=torch.bfloat16, device=a.codes.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = quartz_w4a4_linear_static(_ptr(a.codes), _ptr(a.flags), float(act_scale), _ptr(w.data),
                                   _ptr(bias), _ptr(out), a.M, w.N, a.K, out.stride(0),
                                   a.lzs_group, epilogue, _ptr(workspace), nbytes,
                                   _stream_handle(stream))
    _check(st, "quartz_w4a4_linear_static")
    return out


def weight_group_sums(w: PackedWeight, stream=None):
    """int16 [K/64, N] sums of the int4 weight codes over each 64-group."""
    torch = _torch()
    out = torch.empty((w.K // GROUP, w.N), dtype=torch.int16, device=w.data.device)
    st = quartz_weight_group_sums(_ptr(w.data), w.N, w.K, GROUP, _ptr(out), _stream_handle(stream))
    _check(st, "quartz_weight_group_sums")
    return out


def w4a4_linear_asym(a: QuantizedAct, w: PackedWeight, w_sums, bias=None,
                     epilogue: int = EPI_NONE, out=None, stream=None, workspace=None):
    """Asymmetric-mode layer (quartz_w4a4_linear_asym): ``a`` from quantize_act with
    ``mode=MODE_ASYMMETRIC``, ``w_sums`` from weight_group_sums(w)."""
    torch = _torch()
    _need_mode(a, MODE_ASYMMETRIC, "w4a4_linear_asym")
    if a.K != w.K or a.zeros is None:
        raise ValueError("need asymmetric activations with zero points and matching K")
    if bias is not None and (bias.dtype != torch.bfloat16 or bias.numel() != w.N):
        raise ValueError("bias must be bf16 [N]")
    if out is None:
        out = torch.empty((a.M, w.N), dtype=torch.bfloat16, device=a.codes.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = quartz_w4a4_linear_asym(_ptr(a.codes), _ptr(a.flags), _ptr(a.scales), _ptr(a.zeros),
                                 _ptr(w.data), _ptr(w_sums), _ptr(bias), _ptr(out), a.M, w.N, a.K,
                                 out.stride(0), GROUP, a.lzs_group, epilogue, _ptr(workspace),
                                 nbytes, _stream_handle(stream))
    _check(st, "quartz_w4a4_linear_asym")
    return out


def _conv_args(a: QuantizedAct, w: PackedWeight, images: int, H: int, W: int, bias, out):
    torch = _torch()
    C = a.K
    if a.M != images * H * W:
        raise ValueError("the quantized feature map must have images * H * W rows")
    if w.K != 9 * C:
        raise ValueError("the weight must have K = 9 C (taps (kh, kw), channels fastest)")
    if bias is not None and (bias.dtype != torch.bfloat16 or bias.numel() != w.N):
        raise ValueError("bias must be bf16 [N]")
    if out is None:
        out = torch.empty((a.M, w.N), dtype=torch.bfloat16, device=a.codes.device)
    return C, out


def w4a4_conv3x3(a: QuantizedAct, w: PackedWeight, images: int, H: int, W: int, bias=None,
                 epilogue: int = EPI_NONE, out=None, stream=None, workspace=None):
    """3 x 3 convolution, stride 1, padding 1, as an implicit GEMM
    (quartz_w4a4_conv3x3): ``a`` = quantize_act of the NHWC feature map viewed as
    [images * H * W, C], ``w`` = pack_weight of the weight [N, 9 C] ordered
    (kh, kw, c); returns y bf16 [images * H * W, N] (the workspace from
    ``gemm_workspace(images * H * W, N, 9 C)``)."""
    _need_mode(a, MODE_SYMMETRIC, "w4a4_conv3x3")
    C, out = _conv_args(a, w, images, H, W, bias, out)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = quartz_w4a4_conv3x3(_ptr(a.codes), _ptr(a.flags), _ptr(a.scales), _ptr(w.data),
                             _ptr(bias), _ptr(out), images, H, W, C, w.N, out.stride(0), GROUP,
                             a.lzs_group, epilogue, _ptr(workspace), nbytes,
                             _stream_handle(stream))
    _check(st, "quartz_w4a4_conv3x3")
    return out


def w4a4_conv3x3_static(a: QuantizedAct, w: PackedWeight, act_scale: float, images: int, H: int,
                        W: int, bias=None, epilogue: int = EPI_NONE, out=None, stream=None,
                        workspace=None):
    """The LDM-setting convolution (quartz_w4a4_conv3x3_static): ``a`` =
    quantize_act_static of the feature map with ``act_scale``, ``w`` =
    pack_weight_per_channel of the weight [N, 9 C]."""
    _need_mode(a, MODE_STATIC, "w4a4_conv3x3_static")
    C, out = _conv_args(a, w, images, H, W, bias, out)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = quartz_w4a4_conv3x3_static(_ptr(a.codes), _ptr(a.flags), float(act_scale), _ptr(w.data),
                                    _ptr(bias), _ptr(out), images, H, W, C, w.N, out.stride(0),
                                    a.lzs_group, epilogue, _ptr(workspace), nbytes,
                                    _stream_handle(stream))
    _check(st, "quartz_w4a4_conv3x3_static")
    return out


SCHEDULE_FIELDS = ("tiles_n", "groups", "split", "blocks", "dp_tiles_b0", "sk_first",
                   "sk_tiles", "sk_blocks", "sk_q", "sk_r")
SEGMENT_FIELDS = ("block", "index", "tile", "g0", "g1", "sk_tile", "slot", "b_first", "b_last",
                  "finisher_slot")


def linear_schedule(M: int, N: int, K: int, blocks: int, split: bool = True, tiles: int = 0):
    """Host-side GEMM work schedule for a persistent grid of at most ``blocks``
    workgroups, tiles of 128 x 256 (``tiles=0``, the linear layer) or 256 x 128
    (``tiles=1``, the other GEMM entry points): (dict of SCHEDULE_FIELDS, int32
    numpy array [segments, len(SEGMENT_FIELDS)])."""
    import numpy as np
    sched = np.zeros(len(SCHEDULE_FIELDS), dtype=np.int32)
    n = quartz_w4a4_linear_schedule(M, N, K, blocks, int(split), tiles, sched.ctypes.data, None, 0)
    if n < 0:
        raise ValueError(f"schedule error {n}")
    seg = np.zeros((max(n, 1), len(SEGMENT_FIELDS)), dtype=np.int32)
    n2 = quartz_w4a4_linear_schedule(M, N, K, blocks, int(split), tiles, sched.ctypes.data,
                                     seg.ctypes.data, n)
    assert n2 == n
    return dict(zip(SCHEDULE_FIELDS, (int(v) for v in sched))), seg[:n]


def unpack_weight(w: PackedWeight, stream=None):
    torch = _torch()
    out = torch.empty((w.N, w.K), dtype=torch.int8, device=w.data.device)
    st = quartz_unpack_weight(_ptr(w.data), w.N, w.K, GROUP, _ptr(out), _stream_handle(stream))
    _check(st, "quartz_unpack_weight")
    return out


def w4a4_gemm_i32(a: QuantizedAct, w: PackedWeight, stream=None):
    torch = _torch()
    out = torch.empty((a.M, w.N), dtype=torch.int32, device=a.codes.device)
    st = quartz_w4a4_gemm_i32(_ptr(a.codes), _ptr(a.flags), _ptr(w.data), _ptr(out), a.M, w.N,
                              a.K, GROUP, a.lzs_group, _stream_handle(stream))
    _check(st, "quartz_w4a4_gemm_i32")
    return out


# ------------------------------------------------------------- LZS attention

def quantize_vt(v, heads: int, lzs_group: int = 16, stream=None) -> QuantizedAct:
    """V^T quantized along the keys (quartz_quantize_vt): v bf16 [heads * L, d]
    (rows head * L + key) -> a QuantizedAct with M = heads * d rows (row
    head * d + channel) and K = L."""
    torch = _torch()
    if v.dtype != torch.bfloat16 or v.dim() != 2 or v.stride(1) != 1 or v.shape[0] % heads:
        raise ValueError("v must be a bf16 [heads * L, d] tensor with unit column stride")
    L, d = v.shape[0] // heads, v.shape[1]
    out = _empty_act(heads * d, L, lzs_group, False, v.device)
    st = quartz_quantize_vt(_ptr(v), heads, L, d, v.stride(0), lzs_group, _ptr(out.codes),
                            _ptr(out.flags), _ptr(out.scales), _stream_handle(stream))
    _check(st, "quartz_quantize_vt")
    return out


def attn_scores(q: QuantizedAct, k: QuantizedAct, q_row0: int, k_row0: int, Lq: int, Lk: int,
                scale: float, out=None, stream=None):
    """fp32 scores [Lq, Lk] = scale * Q~ K~^T of one head, the head's rows at
    q_row0 / k_row0 of the quantized queries / keys of all heads."""
    torch = _torch()
    _need_mode(q, MODE_SYMMETRIC, "attn_scores")
    _need_mode(k, MODE_SYMMETRIC, "attn_scores")
    if q.K != k.K or q.lzs_group != k.lzs_group:
        raise ValueError("queries and keys need the same d and G_s")
    if out is None:
        out = torch.empty((Lq, Lk), dtype=torch.float32, device=q.codes.device)
    st = quartz_attn_scores(_ptr(q.codes), _ptr(q.flags), _ptr(q.scales), q.M, q_row0,
                            _ptr(k.codes), _ptr(k.flags), _ptr(k.scales), k.M, k_row0, Lq, Lk,
                            q.K, q.lzs_group, float(scale), _ptr(out), out.stride(0),
                            _stream_handle(stream))
    _check(st, "quartz_attn_scores")
    return out


def softmax_quantize(s, lzs_group: int = 16, out: QuantizedAct | None = None,
                     stream=None) -> QuantizedAct:
    """Row softmax of fp32 scores [M, N] quantized like an activation with K = N."""
    torch = _torch()
    if s.dtype != torch.float32 or s.dim() != 2 or s.stride(1) != 1:
        raise ValueError("s must be a 2-D fp32 tensor with unit column stride")
    M, N = s.shape
    if out is None:
        out = _empty_act(M, N, lzs_group, False, s.device)
    st = quartz_softmax_quantize(_ptr(s), M, N, s.stride(0), lzs_group, _ptr(out.codes),
                                 _ptr(out.flags), _ptr(out.scales), _stream_handle(stream))
    _check(st, "quartz_softmax_quantize")
    return out


def attn_pv(p: QuantizedAct, vt: QuantizedAct, vt_row0: int, d: int, out=None, stream=None,
            workspace=None):
    """bf16 [Lq, d] = P~ V~ of one head: p from softmax_quantize, vt from
    quantize_vt (the head's channels at rows vt_row0 .. vt_row0 + d - 1)."""
    torch = _torch()
    if p.K != vt.K or p.lzs_group != vt.lzs_group:
        raise ValueError("the softmax output and V^T need the same key count and G_s")
    if out is None:
        out = torch.empty((p.M, d), dtype=torch.bfloat16, device=p.codes.device)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = quartz_attn_pv(_ptr(p.codes), _ptr(p.flags), _ptr(p.scales), _ptr(vt.codes),
                        _ptr(vt.flags), _ptr(vt.scales), vt.M, vt_row0, p.M, p.K, d, p.lzs_group,
                        _ptr(out), out.stride(0), _ptr(workspace), nbytes, _stream_handle(stream))
    _check(st, "quartz_attn_pv")
    return out


def attention_workspace(heads: int, L: int, d: int, lzs_group: int, device):
    """Zero-filled workspace of lzs_attention."""
    torch = _torch()
    nbytes = quartz_lzs_attention_workspace_bytes(heads, L, d, lzs_group)
    if nbytes == 0:
        raise ValueError("unsupported attention shape")
    return torch.zeros((nbytes,), dtype=torch.uint8, device=device)


def lzs_attention(q, k, v, heads: int, lzs_group: int = 16, out=None, workspace=None, stream=None):
    """LZS attention of all heads (quartz_lzs_attention): q, k, v bf16
    [heads * L, d] contiguous (head-major); returns bf16 [L, heads * d]."""
    torch = _torch()
    for t in (q, k, v):
        if t.dtype != torch.bfloat16 or t.dim() != 2 or not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous bf16 [heads * L, d] tensors")
    L, d = q.shape[0] // heads, q.shape[1]
    if out is None:
        out = torch.empty((L, heads * d), dtype=torch.bfloat16, device=q.device)
    if workspace is None:
        workspace = attention_workspace(heads, L, d, lzs_group, q.device)
    st = quartz_lzs_attention(_ptr(q), _ptr(k), _ptr(v), heads, L, d, lzs_group, _ptr(out),
                              out.stride(0), _ptr(workspace),
                              workspace.numel() * workspace.element_size(),
                              _stream_handle(stream))
    _check(st, "quartz_lzs_attention")
    return out
