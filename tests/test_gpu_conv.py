"""GPU parity of the implicit 3 x 3 convolution (quartz_w4a4_conv3x3 and
quartz_w4a4_conv3x3_static): the feature map is quantized once on the GPU and
the GEMM reads its codes by tap.  Each case is checked two ways: against the
oracle's layer on the im2col matrix built on the host (within the output
tolerance of tests/helpers.py), and bit for bit against the GPU's explicit
path on that same im2col matrix (quantizer + linear entry point), which by the
reading the host tests pin computes the same codes.  The bit for bit
comparison is between calls without the stream-K split: the linear entry
point runs tiles of another shape, so a split adds its partial sums in
another order; split calls are held to the oracle tolerance.  Ragged images (rows ending inside a tile), several images, C from 64
to 320 (one to five channel blocks), every G_s, GELU, bias, the stream-K
split, a strided output with guard rows, and the config-5 layers at full size
(sampled rows against the oracle)."""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import bf16_bits_to_f64, to_dev_bf16, to_host_u16, y_tolerance

pytestmark = pytest.mark.gpu


def _q():
    import paper_2509_26436_amd as q
    return q


def _fmap(seed, images, H, Wd, C):
    g = np.random.Generator(np.random.PCG64(seed))
    z = g.laplace(0.0, 1.0, size=(images, H, Wd, C))
    x = z / (1.0 + np.exp(-z))
    x[..., g.choice(C, max(1, C // 100), replace=False)] *= 30.0
    return W.to_bf16_bits(x)


def _im2col(fm):
    return np.concatenate([W.im2col3x3(fm[i]) for i in range(fm.shape[0])], axis=0)


def _check(y, y64, S, K, epi):
    err = np.abs(bf16_bits_to_f64(to_host_u16(y)) - y64)
    tol = y_tolerance(y64, S, K, gelu=(epi == 1))
    bad = err > tol
    assert not bad.any(), f"{bad.sum()} outputs out of tolerance; worst excess {(err - tol).max():.3e}"


CASES = [
    # (images, H, W, C, N, gs, epilogue, bias, workspace, pad)
    (1, 9, 9, 64, 72, 16, 0, True, False, 0),
    (2, 17, 13, 128, 130, 8, 1, True, True, 0),
    (1, 20, 20, 192, 64, 32, 0, False, True, 6),
    (3, 8, 8, 64, 200, 64, 0, True, False, 0),
    (1, 16, 33, 320, 96, 16, 0, True, True, 0),
    (1, 1, 5, 64, 64, 16, 0, True, False, 0),        # one image row: every vertical tap pads
]


def _ids(c):
    return f"{c[0]}x{c[1]}x{c[2]}x{c[3]}-N{c[4]}-gs{c[5]}-e{c[6]}{'-ws' if c[8] else ''}"


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_conv_per_group(case):
    import torch
    q = _q()
    images, H, Wd, C, N, gs, epi, with_bias, use_ws, pad = case
    M, K = images * H * Wd, 9 * C
    print(f"conv per-group {case}", flush=True)
    fm = _fmap(M + C + N, images, H, Wd, C)
    cols = _im2col(fm)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 7 + C)).normal(0, 0.02, (N, K)))
    bias_b = W.to_bf16_bits(np.linspace(-0.2, 0.2, N)) if with_bias else None
    bias = None if bias_b is None else to_dev_bf16(bias_b)
    pw = q.pack_weight(to_dev_bf16(wb))
    qa = q.quantize_act(to_dev_bf16(fm.reshape(M, C)), gs)
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    buf = torch.full((M + 64, N + pad), 5.0, dtype=torch.bfloat16, device="cuda")
    y = q.w4a4_conv3x3(qa, pw, images, H, Wd, bias, epi, out=buf[:M, :N], workspace=ws)
    qc = q.quantize_act(to_dev_bf16(cols), gs)
    y_explicit = q.w4a4_linear(qc, pw, bias, epi)
    y_whole = y if ws is None else q.w4a4_conv3x3(qa, pw, images, H, Wd, bias, epi)
    torch.cuda.synchronize()
    assert torch.all(buf[M:] == 5.0) and torch.all(buf[:M, N:] == 5.0), "conv wrote outside y"
    assert torch.equal(y_whole.contiguous().view(torch.int16), y_explicit.view(torch.int16))
    a_ref = oracle.quantize_act(cols, gs)
    wq, sw = oracle.quantize_weight(wb)
    y64, S = oracle.linear_f64(a_ref, wq, sw, bias_b, epilogue=epi)
    _check(y.contiguous(), y64, S, K, epi)


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_conv_static(case):
    import torch
    q = _q()
    images, H, Wd, C, N, gs, epi, with_bias, use_ws, pad = case
    M, K = images * H * Wd, 9 * C
    print(f"conv static {case}", flush=True)
    fm = _fmap(M * 3 + C + N, images, H, Wd, C)
    cols = _im2col(fm)
    s = float(np.float32(np.abs(W.bf16_bits_to_f32(fm)).max() / 127.0 * 0.7))
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 11 + C)).normal(0, 0.02, (N, K)))
    bias_b = W.to_bf16_bits(np.linspace(-0.2, 0.2, N)) if with_bias else None
    bias = None if bias_b is None else to_dev_bf16(bias_b)
    pw = q.pack_weight_per_channel(to_dev_bf16(wb))
    qa = q.quantize_act_static(to_dev_bf16(fm.reshape(M, C)), s, gs)
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    buf = torch.full((M + 64, N + pad), 5.0, dtype=torch.bfloat16, device="cuda")
    y = q.w4a4_conv3x3_static(qa, pw, s, images, H, Wd, bias, epi, out=buf[:M, :N], workspace=ws)
    qc = q.quantize_act_static(to_dev_bf16(cols), s, gs)
    y_explicit = q.w4a4_linear_static(qc, pw, s, bias, epi, workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(buf[M:] == 5.0) and torch.all(buf[:M, N:] == 5.0), "conv wrote outside y"
    assert torch.equal(y.contiguous().view(torch.int16), y_explicit.view(torch.int16))
    a_ref = oracle.quantize_act_static(cols, s, gs)
    wq, sw = oracle.quantize_weight_per_channel(wb)
    y64, S = oracle.linear_static_f64(a_ref, s, wq, sw, bias_b, epi)
    _check(y.contiguous(), y64, S, K, epi)


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_conv_config5_full_size(layer):
    """A config-5 layer at full size in the bench's launch configuration
    (workspace entry point, G_s = 16): the implicit convolution without the
    split bit for bit equal to the explicit GEMM on the host-built im2col
    matrix, and ~60 sampled output pixels of the split call (border and
    interior rows) against the oracle."""
    import torch
    q = _q()
    cfg = 5
    L = W.CONFIGS[cfg].layers[layer]
    C, H = L.K // 9, int(round(L.M ** 0.5))
    print(f"conv full size layer {layer}: {H}x{H}x{C} -> {L.N}", flush=True)
    fm = W.make_feature_map(cfg, layer)
    wb, bias_b = W.make_w(cfg, layer), W.make_bias(cfg, layer)
    pw, bias = q.pack_weight(to_dev_bf16(wb)), to_dev_bf16(bias_b)
    ws = q.gemm_workspace(L.M, L.N, L.K, "cuda")
    qa = q.quantize_act(to_dev_bf16(fm.reshape(L.M, C)), 16)
    y = q.w4a4_conv3x3(qa, pw, 1, H, H, bias, 0, workspace=ws)
    cols = W.make_x(cfg, layer)
    qc = q.quantize_act(to_dev_bf16(cols), 16)
    y_explicit = q.w4a4_linear(qc, pw, bias, 0)
    y_whole = q.w4a4_conv3x3(qa, pw, 1, H, H, bias, 0)
    torch.cuda.synchronize()
    assert torch.equal(y_whole.view(torch.int16), y_explicit.view(torch.int16))
    # the first and last image rows' ends, left and right border pixels of a
    # middle row, and an even spread over the rest
    mid = (H // 2) * H
    rows = np.unique(np.concatenate([np.arange(0, 6), np.arange(H - 3, H + 3), [mid - 1, mid, mid + H - 1],
                                     np.arange(L.M - 6, L.M),
                                     np.linspace(0, L.M - 1, 40).astype(np.int64)]))
    a_ref = oracle.quantize_act(np.ascontiguousarray(cols[rows]), 16)
    wq, sw = oracle.quantize_weight(wb)
    y64, S = oracle.linear_f64(a_ref, wq, sw, bias_b, epilogue=0)
    _check(y[torch.from_numpy(rows).cuda()], y64, S, L.K, 0)


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_conv_static_config5_full_size(layer):
    """The LDM setting of a config-5 layer at full size (workspace entry point,
    G_s = 16, static scale max |x| / 127 of the map): bit for bit equal to the
    explicit static GEMM on the host-built im2col matrix, and sampled pixels
    (border and interior rows) against the oracle."""
    import torch
    q = _q()
    cfg = 5
    L = W.CONFIGS[cfg].layers[layer]
    C, H = L.K // 9, int(round(L.M ** 0.5))
    print(f"static conv full size layer {layer}: {H}x{H}x{C} -> {L.N}", flush=True)
    fm = W.make_feature_map(cfg, layer)
    s = float(np.float32(np.abs(W.bf16_bits_to_f32(fm)).max() / 127.0))
    wb, bias_b = W.make_w(cfg, layer), W.make_bias(cfg, layer)
    pw, bias = q.pack_weight_per_channel(to_dev_bf16(wb)), to_dev_bf16(bias_b)
    ws = q.gemm_workspace(L.M, L.N, L.K, "cuda")
    qa = q.quantize_act_static(to_dev_bf16(fm.reshape(L.M, C)), s, 16)
    y = q.w4a4_conv3x3_static(qa, pw, s, 1, H, H, bias, 0, workspace=ws)
    cols = W.make_x(cfg, layer)
    qc = q.quantize_act_static(to_dev_bf16(cols), s, 16)
    y_explicit = q.w4a4_linear_static(qc, pw, s, bias, 0, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_explicit.view(torch.int16))
    mid = (H // 2) * H
    rows = np.unique(np.concatenate([np.arange(0, 6), np.arange(H - 3, H + 3), [mid - 1, mid, mid + H - 1],
                                     np.arange(L.M - 6, L.M),
                                     np.linspace(0, L.M - 1, 40).astype(np.int64)]))
    a_ref = oracle.quantize_act_static(np.ascontiguousarray(cols[rows]), s, 16)
    wq, sw = oracle.quantize_weight_per_channel(wb)
    y64, S = oracle.linear_static_f64(a_ref, s, wq, sw, bias_b, 0)
    _check(y[torch.from_numpy(rows).cuda()], y64, S, L.K, 0)
