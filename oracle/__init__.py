"""QuaRTZ CPU oracle: test infrastructure only.

A ctypes wrapper over ``quartz_oracle.c`` (plain C, no code shared with the HIP
library).  Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py`` may import this package; the product path never does.

All arrays are numpy arrays.  bf16 and fp16 data travel as ``uint16`` bit
patterns.  See ``quartz_oracle.c`` for the readings of the paper each function
follows (Eq. 1, Eq. 2, Section 3, Section 4.4, Appendices A and C).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "quartz_oracle.c")
_LIB = os.path.join(_HERE, "libquartz_oracle.so")

_lib = None


def build() -> str:
    """Compile the oracle with gcc (IEEE float: no fast-math, no contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-D_DEFAULT_SOURCE", "-ffp-contract=off",
           "-fno-fast-math", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I32 = ctypes.c_int
    lib.qo_bf16_to_f32.argtypes = [ctypes.c_uint16]
    lib.qo_bf16_to_f32.restype = ctypes.c_float
    lib.qo_rne.argtypes = [ctypes.c_double]
    lib.qo_rne.restype = ctypes.c_double
    lib.qo_f16_to_f32.argtypes = [ctypes.c_uint16]
    lib.qo_f16_to_f32.restype = ctypes.c_float
    lib.qo_f32_to_f16_rne_sat.argtypes = [ctypes.c_float]
    lib.qo_f32_to_f16_rne_sat.restype = ctypes.c_uint16
    lib.qo_f64_to_bf16_rne.argtypes = [ctypes.c_double]
    lib.qo_f64_to_bf16_rne.restype = ctypes.c_uint16
    lib.qo_clz32.argtypes = [ctypes.c_uint32]
    lib.qo_clz32.restype = I32
    lib.qo_lzs_flag.argtypes = [ctypes.c_uint32]
    lib.qo_lzs_flag.restype = I32
    lib.qo_gelu_tanh.argtypes = [ctypes.c_double]
    lib.qo_gelu_tanh.restype = ctypes.c_double
    lib.qo_lzs_subgroup.argtypes = [P, I32, P]
    lib.qo_lzs_subgroup.restype = I32
    lib.qo_quantize_act.argtypes = [P, I64, I64, I64, I32, I32, P, P, P, P, P]
    lib.qo_quantize_act.restype = I32
    lib.qo_pack_codes.argtypes = [P, I64, I64, P]
    lib.qo_pack_codes.restype = None
    lib.qo_unpack_codes.argtypes = [P, I64, I64, P]
    lib.qo_unpack_codes.restype = None
    lib.qo_quantize_weight.argtypes = [P, I64, I64, I32, P, P]
    lib.qo_quantize_weight.restype = I32
    lib.qo_gemm_i32.argtypes = [P, P, P, I64, I64, I64, I32, P]
    lib.qo_gemm_i32.restype = I32
    lib.qo_linear_f64.argtypes = [P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, P, P]
    lib.qo_linear_f64.restype = I32
    lib.qo_linear_f64_sampled.argtypes = [P, P, P, P, P, P, I64, I32, I32, I32,
                                          P, P, I64, P, P]
    lib.qo_linear_f64_sampled.restype = I32
    lib.qo_quantize_act_static.argtypes = [P, I64, I64, I64, ctypes.c_float, I32, P, P, P]
    lib.qo_quantize_act_static.restype = I32
    lib.qo_quantize_weight_per_channel.argtypes = [P, I64, I64, P, P]
    lib.qo_quantize_weight_per_channel.restype = I32
    lib.qo_linear_static_f64.argtypes = [P, P, ctypes.c_float, P, P, P, I64, I64, I64, I32, I32,
                                         P, P]
    lib.qo_linear_static_f64.restype = I32
    lib.qo_quantize_act_asym.argtypes = [P, I64, I64, I64, I32, P, P, P, P, P]
    lib.qo_quantize_act_asym.restype = I32
    lib.qo_weight_group_sums.argtypes = [P, I64, I64, P]
    lib.qo_weight_group_sums.restype = I32
    lib.qo_linear_asym_f64.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I32, I32, P, P]
    lib.qo_linear_asym_f64.restype = I32
    lib.qo_quantize_f32.argtypes = [P, I64, I64, I64, I32, P, P, P]
    lib.qo_quantize_f32.restype = I32
    lib.qo_softmax_rows.argtypes = [P, I64, I64, I64, P]
    lib.qo_softmax_rows.restype = I32
    lib.qo_round_bf16.argtypes = [P, I64, P]
    lib.qo_round_bf16.restype = None
    lib.qo_num_threads.argtypes = []
    lib.qo_num_threads.restype = I32
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ scalars

def num_threads() -> int:
    """Threads the oracle's parallel loops use (OpenMP)."""
    return int(_load().qo_num_threads())


def bf16_to_f32(bits: int) -> float:
    return float(_load().qo_bf16_to_f32(int(bits)))


def rne(v: float) -> float:
    return float(_load().qo_rne(float(v)))


def f16_to_f32(bits: int) -> float:
    return float(_load().qo_f16_to_f32(int(bits)))


def f32_to_f16_rne_sat(v: float) -> int:
    return int(_load().qo_f32_to_f16_rne_sat(float(np.float32(v))))


def f64_to_bf16_rne(v: float) -> int:
    return int(_load().qo_f64_to_bf16_rne(float(v)))


def clz32(v: int) -> int:
    return int(_load().qo_clz32(int(v) & 0xFFFFFFFF))


def lzs_flag(m_or: int) -> int:
    return int(_load().qo_lzs_flag(int(m_or) & 0xFFFFFFFF))


def gelu_tanh(v: float) -> float:
    return float(_load().qo_gelu_tanh(float(v)))


def lzs_subgroup(q) -> tuple[int, np.ndarray]:
    """Stage 2 of one subgroup of int8 codes: returns (FLAG, c)."""
    q = _c(q, np.int8)
    c = np.empty_like(q)
    f = _load().qo_lzs_subgroup(_ptr(q), int(q.size), _ptr(c))
    return int(f), c


# --------------------------------------------------------------- arrays

class ActQuant:
    """Oracle outputs of the activation quantizer for x [M][K]."""

    def __init__(self, q8, c, flags, scales, zeros, lzs_group):
        self.q8 = q8          # int8 [M][K]   Stage-1 codes
        self.c = c            # int8 [M][K]   4-bit values in [-7, 7]
        self.flags = flags    # uint8 [M][K/lzs_group]
        self.scales = scales  # uint16 [M][K/64] fp16 bits
        self.zeros = zeros    # int8 [M][K/64]
        self.lzs_group = lzs_group

    @property
    def codes(self) -> np.ndarray:
        """Packed nibbles in the library's storage layout, uint8 [K/64][M][32]."""
        return pack_codes(self.c)

    @property
    def abi_flags(self) -> np.ndarray:
        """Flags in the library's K-group-major layout, uint8 [K/64][M][64/lzs_group]."""
        M, S = self.flags.shape
        per = 64 // self.lzs_group
        return np.ascontiguousarray(self.flags.reshape(M, S // per, per).transpose(1, 0, 2))

    @property
    def abi_scales(self) -> np.ndarray:
        """Scales in the library's K-group-major layout, uint16 [K/64][M]."""
        return np.ascontiguousarray(self.scales.T)

    @property
    def abi_zeros(self) -> np.ndarray:
        return np.ascontiguousarray(self.zeros.T)

    def decoded(self) -> np.ndarray:
        """d = c * 2^FLAG as int32 [M][K]."""
        f = np.repeat(self.flags.astype(np.int32), self.lzs_group, axis=1)
        return self.c.astype(np.int32) << f


def quantize_act(x_bits: np.ndarray, lzs_group: int = 16, group: int = 64,
                 ldx: int | None = None, K: int | None = None) -> ActQuant:
    """x_bits: uint16 bf16 bit patterns [M][ldx] (row-major)."""
    x_bits = _c(x_bits, np.uint16)
    M = x_bits.shape[0]
    ldx = x_bits.shape[1] if ldx is None else ldx
    K = x_bits.shape[1] if K is None else K
    q8 = np.empty((M, K), np.int8)
    c = np.empty((M, K), np.int8)
    flags = np.empty((M, K // lzs_group), np.uint8)
    scales = np.empty((M, K // group), np.uint16)
    zeros = np.empty((M, K // group), np.int8)
    rc = _load().qo_quantize_act(_ptr(x_bits), M, K, ldx, group, lzs_group,
                                 _ptr(q8), _ptr(c), _ptr(flags), _ptr(scales), _ptr(zeros))
    if rc != 0:
        raise ValueError("oracle quantize_act: invalid arguments")
    return ActQuant(q8, c, flags, scales, zeros, lzs_group)


def pack_codes(c: np.ndarray) -> np.ndarray:
    """int8 values [M][K] -> packed nibbles uint8 [K/64][M][32]."""
    c = _c(c, np.int8)
    M, K = c.shape
    out = np.empty((K // 64, M, 32), np.uint8)
    _load().qo_pack_codes(_ptr(c), M, K, _ptr(out))
    return out


def unpack_codes(codes: np.ndarray, M: int, K: int) -> np.ndarray:
    """packed nibbles uint8 [K/64][M][32] -> int8 values [M][K]."""
    codes = _c(codes, np.uint8)
    out = np.empty((M, K), np.int8)
    _load().qo_unpack_codes(_ptr(codes), M, K, _ptr(out))
    return out


def quantize_weight(w_bits: np.ndarray, group: int = 64):
    """w_bits: uint16 bf16 [N][K]; returns (wq int8 [N][K], sw uint16 [N][K/64])."""
    w_bits = _c(w_bits, np.uint16)
    N, K = w_bits.shape
    wq = np.empty((N, K), np.int8)
    sw = np.empty((N, K // group), np.uint16)
    rc = _load().qo_quantize_weight(_ptr(w_bits), N, K, group, _ptr(wq), _ptr(sw))
    if rc != 0:
        raise ValueError("oracle quantize_weight: invalid arguments")
    return wq, sw


def gemm_i32(a: ActQuant, wq: np.ndarray) -> np.ndarray:
    c = _c(a.c, np.int8)
    flags = _c(a.flags, np.uint8)
    wq = _c(wq, np.int8)
    M, K = c.shape
    N = wq.shape[0]
    out = np.empty((M, N), np.int32)
    rc = _load().qo_gemm_i32(_ptr(c), _ptr(flags), _ptr(wq), M, N, K, a.lzs_group, _ptr(out))
    if rc != 0:
        raise ValueError("oracle gemm_i32: invalid arguments")
    return out


def linear_f64(a: ActQuant, wq: np.ndarray, sw: np.ndarray, bias_bits=None,
               epilogue: int = 0, group: int = 64):
    """Returns (y64 float64 [M][N], S float64 [M][N])."""
    c = _c(a.c, np.int8)
    flags = _c(a.flags, np.uint8)
    scales = _c(a.scales, np.uint16)
    wq = _c(wq, np.int8)
    sw = _c(sw, np.uint16)
    bias = None if bias_bits is None else _c(bias_bits, np.uint16)
    M, K = c.shape
    N = wq.shape[0]
    y = np.empty((M, N), np.float64)
    s = np.empty((M, N), np.float64)
    rc = _load().qo_linear_f64(_ptr(c), _ptr(flags), _ptr(scales), _ptr(wq), _ptr(sw),
                               _ptr(bias), M, N, K, group, a.lzs_group, epilogue,
                               _ptr(y), _ptr(s))
    if rc != 0:
        raise ValueError("oracle linear_f64: invalid arguments")
    return y, s


def linear_f64_sampled(a: ActQuant, wq, sw, bias_bits, rows, cols, epilogue: int = 0,
                       group: int = 64):
    """Outputs (rows[i], cols[i]) only: returns (y64 [count], S [count])."""
    c = _c(a.c, np.int8)
    flags = _c(a.flags, np.uint8)
    scales = _c(a.scales, np.uint16)
    wq = _c(wq, np.int8)
    sw = _c(sw, np.uint16)
    bias = None if bias_bits is None else _c(bias_bits, np.uint16)
    rows = _c(rows, np.int64)
    cols = _c(cols, np.int64)
    K = c.shape[1]
    y = np.empty(rows.size, np.float64)
    s = np.empty(rows.size, np.float64)
    rc = _load().qo_linear_f64_sampled(_ptr(c), _ptr(flags), _ptr(scales), _ptr(wq), _ptr(sw),
                                       _ptr(bias), K, group, a.lzs_group, epilogue,
                                       _ptr(rows), _ptr(cols), rows.size, _ptr(y), _ptr(s))
    if rc != 0:
        raise ValueError("oracle linear_f64_sampled: invalid arguments")
    return y, s


def to_bf16_bits(y64: np.ndarray) -> np.ndarray:
    """Expected bf16 output bits (RNE) of float64 values."""
    f = np.vectorize(lambda v: _load().qo_f64_to_bf16_rne(float(v)), otypes=[np.uint16])
    return f(y64)


def round_bf16(y64: np.ndarray) -> np.ndarray:
    """bf16 bits (RNE) of float64 values, same shape; the array form of
    f64_to_bf16_rne."""
    v = _c(y64, np.float64)
    out = np.empty(v.shape, np.uint16)
    _load().qo_round_bf16(_ptr(v), v.size, _ptr(out))
    return out


def linear_quantize(a: ActQuant, wq: np.ndarray, sw: np.ndarray, bias_bits=None,
                    epilogue: int = 0, out_lzs_group: int = 16) -> ActQuant:
    """The layer's output as the next layer's quantized input: the bf16
    output y (linear_f64 rounded to bf16, the value the layer stores) run
    through the activation quantizer with K = N (Eq. 1 and Eq. 2 applied on
    the fly to the producing layer's result, Appendix C)."""
    y64, _ = linear_f64(a, wq, sw, bias_bits, epilogue)
    return quantize_act(round_bf16(y64), out_lzs_group)


# ----------------------------------------------- LDM setting (reading R8)

def quantize_act_static(x_bits: np.ndarray, scale: float, lzs_group: int = 16) -> ActQuant:
    """Static per-tensor quantizer with the fp32 scale ``scale``; the result's
    scales / zeros are None (there are no per-group scales)."""
    x_bits = _c(x_bits, np.uint16)
    M, K = x_bits.shape
    q8 = np.empty((M, K), np.int8)
    c = np.empty((M, K), np.int8)
    flags = np.empty((M, K // lzs_group), np.uint8)
    rc = _load().qo_quantize_act_static(_ptr(x_bits), M, K, K, float(np.float32(scale)), lzs_group,
                                        _ptr(q8), _ptr(c), _ptr(flags))
    if rc != 0:
        raise ValueError("oracle quantize_act_static: invalid arguments")
    return ActQuant(q8, c, flags, None, None, lzs_group)


def quantize_weight_per_channel(w_bits: np.ndarray):
    """w_bits: uint16 bf16 [N][K]; returns (wq int8 [N][K], sw uint16 [N])."""
    w_bits = _c(w_bits, np.uint16)
    N, K = w_bits.shape
    wq = np.empty((N, K), np.int8)
    sw = np.empty(N, np.uint16)
    rc = _load().qo_quantize_weight_per_channel(_ptr(w_bits), N, K, _ptr(wq), _ptr(sw))
    if rc != 0:
        raise ValueError("oracle quantize_weight_per_channel: invalid arguments")
    return wq, sw


def linear_static_f64(a: ActQuant, scale: float, wq: np.ndarray, sw: np.ndarray,
                      bias_bits=None, epilogue: int = 0):
    """LDM-setting layer: returns (y64 float64 [M][N], S float64 [M][N])."""
    c = _c(a.c, np.int8)
    flags = _c(a.flags, np.uint8)
    wq = _c(wq, np.int8)
    sw = _c(sw, np.uint16)
    bias = None if bias_bits is None else _c(bias_bits, np.uint16)
    M, K = c.shape
    N = wq.shape[0]
    y = np.empty((M, N), np.float64)
    s = np.empty((M, N), np.float64)
    rc = _load().qo_linear_static_f64(_ptr(c), _ptr(flags), float(np.float32(scale)), _ptr(wq),
                                      _ptr(sw), _ptr(bias), M, N, K, a.lzs_group, epilogue,
                                      _ptr(y), _ptr(s))
    if rc != 0:
        raise ValueError("oracle linear_static_f64: invalid arguments")
    return y, s


# ------------------------------------------- asymmetric mode (reading R9)

def quantize_act_asym(x_bits: np.ndarray, lzs_group: int = 16) -> ActQuant:
    """Asymmetric quantizer: like quantize_act, with the zero points in ``zeros``."""
    x_bits = _c(x_bits, np.uint16)
    M, K = x_bits.shape
    q8 = np.empty((M, K), np.int8)
    c = np.empty((M, K), np.int8)
    flags = np.empty((M, K // lzs_group), np.uint8)
    scales = np.empty((M, K // 64), np.uint16)
    zeros = np.empty((M, K // 64), np.int8)
    rc = _load().qo_quantize_act_asym(_ptr(x_bits), M, K, K, lzs_group, _ptr(q8), _ptr(c),
                                      _ptr(flags), _ptr(scales), _ptr(zeros))
    if rc != 0:
        raise ValueError("oracle quantize_act_asym: invalid arguments")
    return ActQuant(q8, c, flags, scales, zeros, lzs_group)


def weight_group_sums(wq: np.ndarray) -> np.ndarray:
    """int16 [N][K/64] sums of the int4 weight codes over each 64-group."""
    wq = _c(wq, np.int8)
    N, K = wq.shape
    out = np.empty((N, K // 64), np.int16)
    if _load().qo_weight_group_sums(_ptr(wq), N, K, _ptr(out)) != 0:
        raise ValueError("oracle weight_group_sums: invalid arguments")
    return out


def linear_asym_f64(a: ActQuant, wq: np.ndarray, sw: np.ndarray, bias_bits=None,
                    epilogue: int = 0):
    """Asymmetric-mode layer: returns (y64 float64 [M][N], S float64 [M][N])."""
    c = _c(a.c, np.int8)
    flags = _c(a.flags, np.uint8)
    scales = _c(a.scales, np.uint16)
    zeros = _c(a.zeros, np.int8)
    wq = _c(wq, np.int8)
    sw = _c(sw, np.uint16)
    bias = None if bias_bits is None else _c(bias_bits, np.uint16)
    M, K = c.shape
    N = wq.shape[0]
    y = np.empty((M, N), np.float64)
    s = np.empty((M, N), np.float64)
    rc = _load().qo_linear_asym_f64(_ptr(c), _ptr(flags), _ptr(scales), _ptr(zeros), _ptr(wq),
                                    _ptr(sw), _ptr(bias), M, N, K, a.lzs_group, epilogue,
                                    _ptr(y), _ptr(s))
    if rc != 0:
        raise ValueError("oracle linear_asym_f64: invalid arguments")
    return y, s


# ------------------------------------------------ LZS attention (reading R11)

def quantize_f32(x: np.ndarray, lzs_group: int = 16) -> ActQuant:
    """The activation quantizer on binary32 inputs x [M][K] (float32): the
    form it takes on the softmax output."""
    x = _c(x, np.float32)
    M, K = x.shape
    c = np.empty((M, K), np.int8)
    flags = np.empty((M, K // lzs_group), np.uint8)
    scales = np.empty((M, K // 64), np.uint16)
    rc = _load().qo_quantize_f32(_ptr(x), M, K, K, lzs_group, _ptr(c), _ptr(flags), _ptr(scales))
    if rc != 0:
        raise ValueError("oracle quantize_f32: invalid arguments")
    return ActQuant(None, c, flags, scales, np.zeros((M, K // 64), np.int8), lzs_group)


def softmax_rows(S: np.ndarray) -> np.ndarray:
    """Row softmax of float64 scores, in double, returned as float32."""
    S = _c(S, np.float64)
    M, N = S.shape
    P = np.empty((M, N), np.float32)
    if _load().qo_softmax_rows(_ptr(S), M, N, N, _ptr(P)) != 0:
        raise ValueError("oracle softmax_rows: invalid arguments")
    return P


def _as_operand(a: ActQuant):
    """An LZS-quantized activation used as the second operand of a product:
    its decoded integers c * 2^FLAG (in [-112, 112], so int8) and its fp16
    group scales, in the (wq, sw) form linear_f64 takes."""
    d = a.decoded()
    return d.astype(np.int8), a.scales


def attn_scores_f64(q: ActQuant, k: ActQuant, scale: float, rows=None, cols=None):
    """Scores of one head, S = (Q~ K~^T) * scale with Q~, K~ the quantized
    queries [Lq][d] and keys [Lk][d]: per (i, j) the exact integer products of
    the two 64-groups along d times s_q s_k, summed in double.  With rows /
    cols (index arrays of equal length) only those entries.  Returns (S, A)
    with A = sum_g |s_q s_k P_g| * |scale| (the accumulation's scale)."""
    kd, ks = _as_operand(k)
    if rows is None:
        S, A = linear_f64(q, kd, ks, None)
    else:
        S, A = linear_f64_sampled(q, kd, ks, None, rows, cols)
    return S * scale, A * abs(scale)


def attn_pv_f64(p: ActQuant, vt: ActQuant, rows=None, cols=None):
    """Output of one head from the quantized softmax output P~ [Lq][Lk] and the
    quantized transposed values V~^T [d][Lk] (quantized along the keys):
    O = P~ V~, per (i, c) the exact integer products of the 64-key groups
    times s_p s_v, summed in double.  Returns (O, A) as attn_scores_f64."""
    vd, vs = _as_operand(vt)
    if rows is None:
        return linear_f64(p, vd, vs, None)
    return linear_f64_sampled(p, vd, vs, None, rows, cols)


def lzs_attention_f64(qb, kb, vb, lzs_group: int = 16):
    """One head of LZS attention (reading R11) on bf16 inputs q, k, v [L][d]:
    quantize Q and K along d and V^T along the keys, scores in double, row
    softmax, the softmax output rounded to binary32 and quantized like an
    activation, then O = P~ V~ in double.  Returns (O, parts) with the
    intermediate quantities."""
    d = qb.shape[1]
    qa = quantize_act(qb, lzs_group)
    ka = quantize_act(kb, lzs_group)
    vta = quantize_act(np.ascontiguousarray(np.asarray(vb).T), lzs_group)
    S, _ = attn_scores_f64(qa, ka, 1.0 / np.sqrt(d))
    P = softmax_rows(S)
    pa = quantize_f32(P, lzs_group)
    O, A = attn_pv_f64(pa, vta)
    return O, {"q": qa, "k": ka, "vt": vta, "S": S, "P": P, "p": pa, "A": A}
