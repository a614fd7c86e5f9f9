"""GPU parity of quartz_w4a4_linear_quantize: the layer output quantized in
the GEMM epilogue for the next layer (Eq. 1, Eq. 2 and the right shift of
Section 3, applied on the fly as in Appendix C).

Three kinds of checks:
  * exact inputs (workloads.make_exact_case: power-of-two group scales, so the
    fp32 output is exact and its bf16 rounding unique): codes, flags and
    scales equal the oracle's bit for bit, with and without the stream-K
    workspace, every LZS subgroup size in and out, ragged M, N a multiple of
    64 but not of the 128-column tile;
  * workload-shaped inputs with GELU, where the fp32 output is only known to
    lie within the accumulation bound of the oracle's float64 value: every
    output must be one that some bf16 value in that interval produces (the
    scale, FLAG and code ranges are monotone in the input), and is compared
    exactly wherever that interval admits a single result;
  * the fused output equals quartz_quantize_act of the bf16 output of
    quartz_w4a4_linear(_ws) bit for bit (the same kernel, schedule and
    summation order; only the output code differs).
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import to_dev_bf16, to_host_u16

pytestmark = pytest.mark.gpu


def _q():
    import paper_2509_26436_amd as q
    return q


def _split_of(M, N, K):
    import torch
    q = _q()
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    return q.linear_schedule(M, N, K, blocks)[0]["split"]


def _host(qa):
    """GPU QuantizedAct -> (codes [G][M][32], flags [G][M][FB], scales [G][M] u16, zeros)."""
    z = None if qa.zeros is None else qa.zeros.cpu().numpy()
    return (qa.codes.cpu().numpy(), qa.flags.cpu().numpy(), to_host_u16(qa.scales), z)


def _fused(xb, wb, bias_b, gs, ogs, epi, use_ws, zeros=False):
    import torch
    q = _q()
    qa = q.quantize_act(to_dev_bf16(xb), gs)
    pw = q.pack_weight(to_dev_bf16(wb))
    M, N, K = xb.shape[0], wb.shape[0], xb.shape[1]
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    bias = None if bias_b is None else to_dev_bf16(bias_b)
    out = q.w4a4_linear_quantize(qa, pw, bias, epi, ogs, with_zeros=zeros, workspace=ws)
    torch.cuda.synchronize()
    return qa, pw, bias, ws, out


EXACT = [
    # (M, N, K, gs, out_gs, bias, workspace, zeros)
    (300, 320, 256, 16, 16, True, False, True),     # ragged M, half-used last column tile
    (300, 320, 2048, 8, 32, True, True, False),     # split along K (tiles shared)
    (64, 64, 128, 64, 8, False, False, False),      # one wave column
    (1, 128, 2048, 32, 64, True, True, False),      # a single row, one tile over 2 workgroups
    (513, 448, 2048, 16, 16, True, True, True),     # three tile rows, split
    (256, 1152, 512, 16, 16, True, False, False),   # the single-linear width
]


@pytest.mark.parametrize("case", EXACT, ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}-gs{c[3]}-o{c[4]}"
                         f"{'-ws' if c[6] else ''}")
def test_exact_inputs_bit_exact(case):
    M, N, K, gs, ogs, with_bias, use_ws, zeros = case
    print(f"fused quantize exact M={M} N={N} K={K} gs={gs} out_gs={ogs} ws={use_ws}", flush=True)
    if use_ws:
        assert _split_of(M, N, K) == 1
    c = W.make_exact_case(7000 + M + N + K, M, N, K)
    bias_b = c.bias if with_bias else None
    _, _, _, _, out = _fused(c.x, c.w, bias_b, gs, ogs, 0, use_ws, zeros)
    a_ref = oracle.quantize_act(c.x, gs)
    wq, sw = oracle.quantize_weight(c.w)
    ref = oracle.linear_quantize(a_ref, wq, sw, bias_b, 0, ogs)
    codes, flags, scales, z = _host(out)
    np.testing.assert_array_equal(scales, ref.abi_scales)
    np.testing.assert_array_equal(flags, ref.abi_flags)
    np.testing.assert_array_equal(codes, ref.codes)
    if zeros:
        assert np.all(z == 0)


def _flag_table():
    return np.array([oracle.lzs_flag(m) for m in range(128)], np.int64)


def _check_admissible(out, y64, S, K, gelu, ogs):
    """Every output is the quantization of some bf16 vector within the error
    bound of the oracle's float64 output; returns the fraction of codes that
    bound determines uniquely."""
    M, N = y64.shape
    G = N // 64
    tol = 4.0 * (K / 64 + 1) * 2.0 ** -24 * S
    if gelu:
        # the GELU slope stays below 1.13; its fp32 evaluation adds a relative
        # error of a few units of 2^-20 at most
        tol = 1.2 * tol + 2.0 ** -14 * np.abs(y64)
    vlo = W.bf16_bits_to_f32(oracle.round_bf16(y64 - tol)).astype(np.float64)
    vhi = W.bf16_bits_to_f32(oracle.round_bf16(y64 + tol)).astype(np.float64)
    spans0 = (vlo <= 0) & (vhi >= 0)
    amin = np.where(spans0, 0.0, np.minimum(np.abs(vlo), np.abs(vhi)))
    amax = np.maximum(np.abs(vlo), np.abs(vhi))
    codes, flags, scales, _ = _host(out)
    c_gpu = oracle.unpack_codes(codes, M, N).astype(np.int64)             # [M][N]
    s_gpu = scales.T                                                      # [M][G] u16
    # scale: fp16(alpha / 127) is monotone in alpha
    a_lo = amin.reshape(M, G, 64).max(axis=2).astype(np.float32)
    a_hi = amax.reshape(M, G, 64).max(axis=2).astype(np.float32)
    s_lo = (a_lo / np.float32(127)).astype(np.float16).view(np.uint16)
    s_hi = (a_hi / np.float32(127)).astype(np.float16).view(np.uint16)
    assert np.all((s_gpu >= s_lo) & (s_gpu <= s_hi)), "scale outside its admissible range"
    # |q| range with the GPU's scale
    s = s_gpu.view(np.float16).astype(np.float32)
    r = np.where(s == 0, np.float32(0), np.float32(1) / np.where(s == 0, np.float32(1), s))
    rr = np.repeat(r, 64, axis=1)
    q_lo = np.minimum(np.rint(amin.astype(np.float32) * rr), 127).astype(np.int64)
    q_hi = np.minimum(np.rint(amax.astype(np.float32) * rr), 127).astype(np.int64)
    # FLAG = max over the subgroup of flag(|q|), monotone in each |q|
    ft = _flag_table()
    nsub = N // ogs
    f_lo = ft[q_lo].reshape(M, nsub, ogs).max(axis=2)
    f_hi = ft[q_hi].reshape(M, nsub, ogs).max(axis=2)
    f_gpu = flags.transpose(1, 0, 2).reshape(M, nsub).astype(np.int64)
    assert np.all((f_gpu >= f_lo) & (f_gpu <= f_hi)), "FLAG outside its admissible range"
    F = np.repeat(f_gpu, ogs, axis=1)
    mag = np.abs(c_gpu)
    assert np.all((mag >= (q_lo >> F)) & (mag <= (q_hi >> F))), "code magnitude not admissible"
    neg_ok = (vlo < 0)
    pos_ok = (vhi > 0)
    assert np.all((c_gpu == 0) | ((c_gpu > 0) & pos_ok) | ((c_gpu < 0) & neg_ok)), "code sign"
    unique = (s_lo == s_hi).repeat(64, axis=1) & (np.repeat(f_lo == f_hi, ogs, axis=1)) & \
             ((q_lo >> F) == (q_hi >> F)) & ~spans0
    return float(unique.mean())


REAL = [
    # (cfg, layer, M, N, gs, out_gs, epilogue, workspace)
    (3, 2, 300, 1152, 16, 16, 1, True),     # FLUX fc1 rows, GELU, split
    (2, 2, 257, 1216, 8, 32, 1, False),     # PixArt fc1 rows, ragged M, half tile
    (1, 0, 96, 640, 32, 8, 0, True),        # single linear, no activation
]


@pytest.mark.parametrize("case", REAL, ids=lambda c: f"cfg{c[0]}l{c[1]}-{c[2]}x{c[3]}-o{c[5]}")
def test_workload_outputs_admissible(case):
    cfg, layer, M, N, gs, ogs, epi, use_ws = case
    L = W.CONFIGS[cfg].layers[layer]
    K = L.K
    print(f"fused quantize workload cfg={cfg} layer={layer} M={M} N={N} K={K}", flush=True)
    xb = W.make_x(cfg, layer, rows=M)
    wb = W.make_w(cfg, layer, rows=N)
    bias_b = W.make_bias(cfg, layer, cols=N)
    _, _, _, _, out = _fused(xb, wb, bias_b, gs, ogs, epi, use_ws)
    a_ref = oracle.quantize_act(xb, gs)
    wq, sw = oracle.quantize_weight(wb)
    y64, S = oracle.linear_f64(a_ref, wq, sw, bias_b, epilogue=epi)
    frac = _check_admissible(out, y64, S, K, epi == 1, ogs)
    print(f"codes determined by the bound: {frac:.4f}", flush=True)
    assert frac > 0.5


def test_tiny_outputs_take_the_clamped_path():
    """Weights scaled down so that the output groups get subnormal fp16 scales
    (the case where the clamp to 127 can bind)."""
    M, N, K = 128, 256, 1152
    xb = W.make_x(1, 0, rows=M)
    w = W.bf16_bits_to_f32(W.make_w(1, 0, rows=N)).astype(np.float64) * 1e-4
    wb = W.to_bf16_bits(w)
    _, _, _, _, out = _fused(xb, wb, None, 16, 16, 0, False)
    a_ref = oracle.quantize_act(xb, 16)
    wq, sw = oracle.quantize_weight(wb)
    y64, S = oracle.linear_f64(a_ref, wq, sw, None)
    s = to_host_u16(out.scales)
    assert np.any((s > 0) & (s < 0x0400)), "no subnormal scale reached"
    _check_admissible(out, y64, S, K, False, 16)


@pytest.mark.parametrize("use_ws", [False, True])
@pytest.mark.parametrize("ogs", [8, 64])
def test_equals_quantizing_the_stored_output(use_ws, ogs):
    import torch
    q = _q()
    cfg, layer, M, N = 3, 2, 600, 1536
    print(f"fused vs unfused cfg={cfg} layer={layer} M={M} N={N} ws={use_ws} out_gs={ogs}", flush=True)
    xb = W.make_x(cfg, layer, rows=M)
    wb = W.make_w(cfg, layer, rows=N)
    bias_b = W.make_bias(cfg, layer, cols=N)
    qa, pw, bias, ws, out = _fused(xb, wb, bias_b, 16, ogs, 1, use_ws)
    y = q.w4a4_linear(qa, pw, bias, 1, workspace=ws)
    ref = q.quantize_act(y, ogs)
    torch.cuda.synchronize()
    for a, b in zip(_host(out)[:3], _host(ref)[:3]):
        np.testing.assert_array_equal(a, b)
    # a second call on the same workspace gives the same bits
    again = q.w4a4_linear_quantize(qa, pw, bias, 1, ogs, workspace=ws)
    torch.cuda.synchronize()
    for a, b in zip(_host(out)[:3], _host(again)[:3]):
        np.testing.assert_array_equal(a, b)


def test_zero_activations():
    import torch
    q = _q()
    M, N, K = 70, 128, 256
    xb = np.zeros((M, K), np.uint16)
    wb = W.make_w(1, 0, rows=N)[:, :K].copy()
    qa = q.quantize_act(to_dev_bf16(xb), 16)
    pw = q.pack_weight(to_dev_bf16(wb))
    out = q.w4a4_linear_quantize(qa, pw, None, 0, 16)
    torch.cuda.synchronize()
    codes, flags, scales, _ = _host(out)
    assert not codes.any() and not flags.any() and not scales.any()


def test_full_size_batched_mlp_fc1_equals_quantizing_the_stored_output():
    """The batched FLUX MLP's fc1 (M = 18432, K = 3072, N = 12288, GELU) at full
    size through the workspace entry point, as the bench times it: every
    code, FLAG and scale of the fused output equals the quantizer applied to
    the layer's stored bf16 output (whose parity with the oracle the
    full-size pipeline test checks on sampled rows)."""
    import torch
    q = _q()
    L = W.CONFIGS[4].layers[0]
    print(f"fused vs unfused full size M={L.M} K={L.K} N={L.N}", flush=True)
    qa, pw, bias, ws, out = _fused(W.make_x(4, 0), W.make_w(4, 0), W.make_bias(4, 0), 16, 16,
                                   L.epilogue, True)
    y = q.w4a4_linear(qa, pw, bias, L.epilogue, workspace=ws)
    ref = q.quantize_act(y, 16)
    torch.cuda.synchronize()
    for name, a, b in zip(("codes", "flags", "scales"), (out.codes, out.flags, out.scales),
                          (ref.codes, ref.flags, ref.scales)):
        assert torch.equal(a, b), f"fused {name} differ from quantizing the stored output"
