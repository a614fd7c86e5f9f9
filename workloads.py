"""Seeded synthetic workloads for the QuaRTZ W4A4 linear path.

This module only draws inputs: layer shapes and activation / weight / bias
tensors with the distributions of diffusion-model linear layers (DiT and
UNet-conv-as-GEMM shapes at the paper's model families, Section 5.1).  It holds
none of the method's arithmetic (no quantization, no LZS, no GEMM), so both the
CPU oracle and the HIP path can consume its outputs.

Every tensor is drawn with numpy's PCG64 in float64, cast to float32 and then to
bf16 with round-to-nearest-even; bf16 tensors are returned as uint16 bit
patterns.  Seeds: ``250926436 + 100*config + 10*layer + tensor`` with tensor
0 = x, 1 = w, 2 = bias, 3 = outlier-channel choice.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 250926436


@dataclass(frozen=True)
class Layer:
    name: str
    M: int
    K: int
    N: int
    x_kind: str            # activation recipe, see make_x()
    w_std: float
    epilogue: int = 0      # 0 = none, 1 = GELU-tanh
    bias: bool = True


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    layers: tuple = field(default_factory=tuple)


CONFIGS = {
    1: Config(1, "single_linear_m256_k1152_n1152", (
        Layer("linear", 256, 1152, 1152, "laplace_0.05_out0.5pct_x30", 0.02),
    )),
    2: Config(2, "pixart_sigma_1024px_block", (
        Layer("qkv", 4096, 1152, 3456, "laplace_0.1_out1pct_u1_50", 0.02),
        Layer("proj", 4096, 1152, 1152, "laplace_0.1_out1pct_u1_50", 0.02),
        Layer("fc1", 4096, 1152, 4608, "laplace_0.1_out1pct_u1_50", 0.02),
        Layer("fc2", 4096, 4608, 1152, "post_gelu_clip_-0.17", 0.02),
    )),
    3: Config(3, "flux1_schnell_joint_block_m4608", (
        Layer("qkv", 4608, 3072, 9216, "t3_0.05_out0.2pct_x100", 0.015),
        Layer("out", 4608, 3072, 3072, "t3_0.05_out0.2pct_x100", 0.015),
        Layer("fc1", 4608, 3072, 12288, "t3_0.05_out0.2pct_x100", 0.015),
        Layer("fc2", 4608, 12288, 3072, "post_gelu_t3", 0.015),
    )),
    4: Config(4, "flux_mlp_batched_m18432", (
        Layer("fc1", 18432, 3072, 12288, "t3_0.05_out0.2pct_x100", 0.015, epilogue=1),
        Layer("fc2", 18432, 12288, 3072, "pipeline", 0.015),
    )),
    5: Config(5, "sdxl_unet_conv3x3_im2col", (
        Layer("conv128x128x320", 16384, 2880, 320, "im2col_silu_c320_h128", 0.02),
        Layer("conv64x64x640", 4096, 5760, 640, "im2col_silu_c640_h64", 0.02),
        Layer("conv32x32x1280", 1024, 11520, 1280, "im2col_silu_c1280_h32", 0.02),
    )),
}


def seed(config: int, layer: int, tensor: int) -> int:
    return SEED_BASE + 100 * config + 10 * layer + tensor


def rng(config: int, layer: int, tensor: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed(config, layer, tensor)))


def to_bf16_bits(a) -> np.ndarray:
    """float64/float32 array -> bf16 bit patterns (float32 first, then RNE)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    # round to nearest even on the 16 dropped bits (no overflow for finite values)
    r = (u >> 16) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _gelu_tanh_np(z):
    """0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))), evaluated in place."""
    t = z * z
    t *= z
    t *= 0.044715
    t += z
    t *= np.sqrt(2.0 / np.pi)
    np.tanh(t, out=t)
    t += 1.0
    t *= z
    t *= 0.5
    return t


def _outlier_cols(config: int, layer: int, K: int, frac: float,
                  g3: np.random.Generator | None = None) -> np.ndarray:
    n = max(1, int(round(frac * K)))
    g3 = rng(config, layer, 3) if g3 is None else g3
    return g3.choice(K, n, replace=False)


def make_x(config: int, layer_index: int, rows: int | None = None) -> np.ndarray:
    """Activation x [rows][K] as bf16 bits.  ``rows`` truncates M (same recipe,
    same leading rows as the full tensor)."""
    L = CONFIGS[config].layers[layer_index]
    M = L.M if rows is None else rows
    K = L.K
    g = rng(config, layer_index, 0)
    kind = L.x_kind
    if kind == "laplace_0.05_out0.5pct_x30":
        x = g.laplace(0.0, 0.05, size=(M, K))
        x[:, _outlier_cols(config, layer_index, K, 0.005)] *= 30.0
    elif kind == "laplace_0.1_out1pct_u1_50":
        x = g.laplace(0.0, 0.1, size=(M, K))
        g3 = rng(config, layer_index, 3)
        cols = _outlier_cols(config, layer_index, K, 0.01, g3)
        x[:, cols] *= g3.uniform(1.0, 50.0, size=cols.size)
    elif kind == "post_gelu_clip_-0.17":
        z = g.laplace(0.0, 0.1, size=(M, K))
        g3 = rng(config, layer_index, 3)
        cols = _outlier_cols(config, layer_index, K, 0.01, g3)
        z[:, cols] *= g3.uniform(1.0, 50.0, size=cols.size)
        x = _gelu_tanh_np(z)
        np.maximum(x, -0.17, out=x)
    elif kind == "t3_0.05_out0.2pct_x100":
        x = g.standard_t(3.0, size=(M, K))
        x *= 0.05
        x[:, _outlier_cols(config, layer_index, K, 0.002)] *= 100.0
    elif kind == "post_gelu_t3":
        z = g.standard_t(3.0, size=(M, K))
        z *= 0.05
        z[:, _outlier_cols(config, layer_index, K, 0.002)] *= 100.0
        x = _gelu_tanh_np(z)
    elif kind == "pipeline":
        raise ValueError("the fc2 input of the batched MLP is fc1's output")
    elif kind.startswith("im2col_silu_"):
        x = _im2col_silu(config, layer_index, M, K, kind)
    else:
        raise ValueError(kind)
    return to_bf16_bits(x)


def _conv_shape(kind):
    """(C, H) of an im2col_silu_c<C>_h<H> layer (square feature map H x H)."""
    parts = kind.split("_")
    return int(parts[2][1:]), int(parts[3][1:])


def _feature_map(config, layer_index, img_rows, H, C):
    """The first img_rows rows of the layer's H x H x C feature map (NHWC,
    float64): SiLU(Laplace(0, 1)) with 0.5% of the C input channels x30."""
    g = rng(config, layer_index, 0)
    z = g.laplace(0.0, 1.0, size=(img_rows, H, C))
    fmap = z / (1.0 + np.exp(-z))
    fmap[:, :, _outlier_cols(config, layer_index, C, 0.005)] *= 30.0
    return fmap


def im2col3x3(fmap: np.ndarray, rows: int | None = None) -> np.ndarray:
    """im2col of a 3 x 3 convolution, stride 1, padding 1, of one feature map
    [Hs, W, C] (any dtype): row r = output pixel (r // W, r % W), K = 9 C
    ordered (kh, kw, c) with c fastest; taps outside the map (or past its Hs
    rows) read zero.  ``rows`` truncates to the first output pixels."""
    Hs, W, C = fmap.shape
    M = Hs * W if rows is None else rows
    out = np.zeros((M, 9 * C), dtype=fmap.dtype)
    oy, ox = np.divmod(np.arange(M), W)
    for kh in range(3):
        for kw in range(3):
            iy, ix = oy + kh - 1, ox + kw - 1
            ok = (iy >= 0) & (iy < Hs) & (ix >= 0) & (ix < W)
            t = kh * 3 + kw
            out[ok, t * C:(t + 1) * C] = fmap[iy[ok], ix[ok]]
    return out


def make_feature_map(config: int, layer_index: int, img_rows: int | None = None) -> np.ndarray:
    """The NHWC feature map [img_rows][W][C] of a config-5 layer as bf16 bits;
    make_x(config, layer) is its im2col (same values, same leading rows)."""
    L = CONFIGS[config].layers[layer_index]
    C, H = _conv_shape(L.x_kind)
    return to_bf16_bits(_feature_map(config, layer_index, H if img_rows is None else img_rows, H, C))


def _im2col_silu(config, layer_index, M, K, kind):
    """3x3 conv (padding 1) as GEMM: rows are output pixels, K = 9*C ordered
    (kh, kw, c) with c fastest; the feature map is SiLU(Laplace(0, 1)) with
    0.5% of the C input channels x30; border taps read zero padding."""
    C, H = _conv_shape(kind)
    assert K == 9 * C
    n_img_rows = min(H, (M + H - 1) // H + 1)
    return im2col3x3(_feature_map(config, layer_index, n_img_rows, H, C), rows=M)


def make_w(config: int, layer_index: int, rows: int | None = None) -> np.ndarray:
    """Weight w [N][K] (nn.Linear layout) as bf16 bits."""
    L = CONFIGS[config].layers[layer_index]
    N = L.N if rows is None else rows
    x = rng(config, layer_index, 1).normal(0.0, L.w_std, size=(N, L.K))
    return to_bf16_bits(x)


def make_bias(config: int, layer_index: int, cols: int | None = None) -> np.ndarray:
    L = CONFIGS[config].layers[layer_index]
    N = L.N if cols is None else cols
    return to_bf16_bits(rng(config, layer_index, 2).normal(0.0, 0.02, size=N))


def make_random_x(seed_value: int, M: int, K: int, kind: str = "laplace",
                  scale: float = 0.1) -> np.ndarray:
    """Free-form seeded activations for edge-case tests."""
    g = np.random.Generator(np.random.PCG64(seed_value))
    if kind == "laplace":
        x = g.laplace(0.0, scale, size=(M, K))
    elif kind == "normal":
        x = g.normal(0.0, scale, size=(M, K))
    elif kind == "t3":
        x = scale * g.standard_t(3.0, size=(M, K))
    else:
        raise ValueError(kind)
    return to_bf16_bits(x)


@dataclass(frozen=True)
class ExactCase:
    """Inputs whose layer output is exact in fp32 (see make_exact_case)."""
    A: np.ndarray          # int64 [M][K], |A| <= 127, a +-127 in every 64-group of a row
    Wi: np.ndarray         # int64 [N][K], |Wi| <= 7, a +-7 in every 64-group of a row
    e: np.ndarray          # int64 [M]: row m of x is A[m] * 2^e[m]
    f: np.ndarray          # int64 [N]: row n of w is Wi[n] * 2^f[n]
    x: np.ndarray          # bf16 bits [M][K]
    w: np.ndarray          # bf16 bits [N][K]
    bias: np.ndarray       # bf16 bits [N]: b_int[n] * 2^(f[n] + max e)
    bias_val: np.ndarray   # float64 [N]


def _int_rows(g: np.random.Generator, rows: int, K: int, top: int) -> np.ndarray:
    a = g.integers(-top, top + 1, size=(rows, K)).astype(np.int64)
    for k0 in range(0, K, 64):
        pos = g.integers(0, 64, size=rows)
        sign = np.where(g.integers(0, 2, size=rows) == 1, 1, -1)
        a[np.arange(rows), k0 + pos] = top * sign
    return a


def make_exact_case(seed_value: int, M: int, N: int, K: int) -> ExactCase:
    """Activations A * 2^e (integers up to 127 with a +-127 in every 64-group)
    and weights Wi * 2^f (integers up to 7 with a +-7 in every 64-group): every
    group's max |x| / 127 and max |w| / 7 is a power of two, and the bias is an
    integer of at most 8 bits times 2^(f + max e).  Any sum of products of such
    values with scales 2^e, 2^f is an integer times 2^(e + f); for K up to a
    few thousand it stays below 2^24 of that unit, i.e. exact in fp32."""
    g = np.random.Generator(np.random.PCG64(seed_value))
    A = _int_rows(g, M, K, 127)
    Wi = _int_rows(g, N, K, 7)
    e = g.integers(-6, -1, size=M)
    f = g.integers(-9, -4, size=N)
    x = to_bf16_bits(np.ldexp(A.astype(np.float64), e[:, None]))
    w = to_bf16_bits(np.ldexp(Wi.astype(np.float64), f[:, None]))
    b_int = g.integers(-255, 256, size=N)
    bias_val = np.ldexp(b_int.astype(np.float64), f + e.max())
    return ExactCase(A, Wi, e, f, x, w, to_bf16_bits(bias_val), bias_val)
