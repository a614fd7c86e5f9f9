"""GPU parity of the LDM setting (the paper's experimental-details appendix:
static per-tensor activation quantization, per-channel weight quantization,
4-bit LZS on the fly; reading R8): quartz_quantize_act_static and
quartz_pack_weight_per_channel bit-exact against the oracle, the exact
integer accumulator of their outputs, and quartz_w4a4_linear_static within
the output tolerance of tests/helpers.py, with and without the stream-K
workspace, at small ragged shapes and at a full FLUX layer (sampled rows)."""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import bf16_bits_to_f64, to_dev_bf16, to_host_u16, y_tolerance

pytestmark = pytest.mark.gpu


def _q():
    import paper_2509_26436_amd as q
    return q


def _calibrated_scale(xb, frac=0.6):
    """A static scale below the tensor's own range, so some values clip."""
    return float(np.float32(np.abs(W.bf16_bits_to_f32(xb)).max() / 127.0 * frac))


@pytest.mark.parametrize("gs", [8, 16, 32, 64])
@pytest.mark.parametrize("cfg,layer,M", [(1, 0, 200), (3, 3, 37), (5, 0, 129), (2, 3, 1)])
def test_static_quantizer_bit_exact(cfg, layer, M, gs):
    import torch
    q = _q()
    xb = W.make_x(cfg, layer, rows=M)
    s = _calibrated_scale(xb)
    print(f"static quantize cfg={cfg} layer={layer} M={M} gs={gs} s={s}", flush=True)
    qa = q.quantize_act_static(to_dev_bf16(xb), s, gs)
    torch.cuda.synchronize()
    ref = oracle.quantize_act_static(xb, s, gs)
    np.testing.assert_array_equal(qa.flags.cpu().numpy(), ref.abi_flags)
    np.testing.assert_array_equal(qa.codes.cpu().numpy(), ref.codes)
    assert np.any(np.abs(ref.q8) == 127)


def test_static_quantizer_strided_rows():
    import torch
    q = _q()
    M, K = 70, 576
    xb = W.make_random_x(5, M, K + 40, "laplace", 0.1)
    s = _calibrated_scale(xb[:, :K], 0.8)
    x = to_dev_bf16(xb)[:, :K]
    qa = q.quantize_act_static(x, s, 16)
    torch.cuda.synchronize()
    ref = oracle.quantize_act_static(np.ascontiguousarray(xb[:, :K]), s, 16)
    np.testing.assert_array_equal(qa.codes.cpu().numpy(), ref.codes)
    np.testing.assert_array_equal(qa.flags.cpu().numpy(), ref.abi_flags)


@pytest.mark.parametrize("N,K", [(136, 192), (64, 64), (1, 128), (320, 2880), (1152, 4608)])
def test_per_channel_pack_bit_exact(N, K):
    import torch
    q = _q()
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 3 + K)).normal(0, 0.02, (N, K)))
    print(f"per-channel pack N={N} K={K}", flush=True)
    pw = q.pack_weight_per_channel(to_dev_bf16(wb))
    wq = q.unpack_weight(pw)
    torch.cuda.synchronize()
    wq_ref, sw_ref = oracle.quantize_weight_per_channel(wb)
    np.testing.assert_array_equal(to_host_u16(pw.scales), sw_ref)
    np.testing.assert_array_equal(wq.cpu().numpy(), wq_ref)
    # every group's scale slot holds the channel scale; padding columns are zero
    G = K // 64
    panels = (N + 63) // 64
    raw = pw.data.cpu().numpy()[:panels * G * 2176].reshape(panels, G, 2176)
    slots = raw[:, :, 2048:].copy().view(np.uint16).reshape(panels, G, 64)
    col = np.zeros(panels * 64, np.uint16)
    col[:N] = sw_ref
    np.testing.assert_array_equal(slots, np.broadcast_to(col.reshape(panels, 1, 64), slots.shape))
    codes = raw[:, :, :2048].reshape(panels, G, 64, 32)
    if N % 64:
        assert not codes[-1, :, N % 64:, :].any()


def _ldm_case(xb, wb, gs):
    q = _q()
    s = _calibrated_scale(xb)
    qa = q.quantize_act_static(to_dev_bf16(xb), s, gs)
    pw = q.pack_weight_per_channel(to_dev_bf16(wb))
    a_ref = oracle.quantize_act_static(xb, s, gs)
    wq_ref, sw_ref = oracle.quantize_weight_per_channel(wb)
    return s, qa, pw, a_ref, wq_ref, sw_ref


@pytest.mark.parametrize("gs", [8, 16, 32, 64])
@pytest.mark.parametrize("M,N,K", [(200, 136, 192), (129, 129, 128), (256, 384, 1152)])
def test_static_integer_accumulator(M, N, K, gs):
    import torch
    q = _q()
    xb = W.make_random_x(M * 11 + N, M, K, "t3", 0.05)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N + 5 * K)).normal(0, 0.02, (N, K)))
    _, qa, pw, a_ref, wq_ref, _ = _ldm_case(xb, wb, gs)
    acc = q.w4a4_gemm_i32(qa, pw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(acc.cpu().numpy(), oracle.gemm_i32(a_ref, wq_ref))


def _check(y, y64, S, K, epi):
    err = np.abs(bf16_bits_to_f64(to_host_u16(y)) - y64)
    tol = y_tolerance(y64, S, K, gelu=(epi == 1))
    bad = err > tol
    assert not bad.any(), f"{bad.sum()} outputs out of tolerance; worst excess {(err - tol).max():.3e}"


CASES = [
    # (cfg, layer, M, N, gs, epilogue, bias, workspace, ldy_pad)
    (1, 0, 200, 136, 16, 0, True, False, 0),
    (2, 3, 160, 448, 16, 1, True, True, 0),       # K = 4608, split along K
    (3, 0, 300, 200, 8, 0, False, True, 6),       # ragged, no bias, strided output
    (3, 3, 257, 129, 32, 0, True, True, 0),       # K = 12288, split
    (5, 1, 64, 640, 64, 1, True, False, 0),       # K = 5760, GELU
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"cfg{c[0]}l{c[1]}-{c[2]}x{c[3]}-gs{c[4]}"
                         f"{'-ws' if c[7] else ''}")
def test_static_linear_parity(case):
    import torch
    q = _q()
    cfg, layer, M, N, gs, epi, with_bias, use_ws, pad = case
    K = W.CONFIGS[cfg].layers[layer].K
    print(f"static linear cfg={cfg} layer={layer} M={M} N={N} K={K} gs={gs} ws={use_ws}", flush=True)
    xb = W.make_x(cfg, layer, rows=M)
    wb = W.make_w(cfg, layer, rows=N)
    bias_b = W.make_bias(cfg, layer, cols=N) if with_bias else None
    s, qa, pw, a_ref, wq_ref, sw_ref = _ldm_case(xb, wb, gs)
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    bias = None if bias_b is None else to_dev_bf16(bias_b)
    if pad:
        ybuf = torch.full((M, N + pad), 3.0, dtype=torch.bfloat16, device="cuda")
        q.w4a4_linear_static(qa, pw, s, bias, epi, out=ybuf[:, :N], workspace=ws)
        torch.cuda.synchronize()
        assert torch.all(ybuf[:, N:] == 3.0)
        y = ybuf[:, :N].contiguous()
    else:
        y = q.w4a4_linear_static(qa, pw, s, bias, epi, workspace=ws)
        torch.cuda.synchronize()
    y64, S = oracle.linear_static_f64(a_ref, s, wq_ref, sw_ref, bias_b, epi)
    _check(y, y64, S, K, epi)
    if use_ws:
        again = q.w4a4_linear_static(qa, pw, s, bias, epi, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(again.view(torch.int16), y.view(torch.int16))


def test_static_linear_full_flux_layer_sampled_rows():
    """The FLUX out projection at full size (M = 4608, K = N = 3072) through
    the workspace entry point; 96 rows spread over every tile row compared with
    the oracle (static quantization is row-local)."""
    import torch
    q = _q()
    cfg, layer = 3, 1
    L = W.CONFIGS[cfg].layers[layer]
    print(f"static linear full size {L.M}x{L.N}x{L.K}", flush=True)
    xb = W.make_x(cfg, layer)
    wb = W.make_w(cfg, layer)
    bias_b = W.make_bias(cfg, layer)
    s = _calibrated_scale(xb, 0.9)
    qa = q.quantize_act_static(to_dev_bf16(xb), s, 16)
    pw = q.pack_weight_per_channel(to_dev_bf16(wb))
    ws = q.gemm_workspace(L.M, L.N, L.K, "cuda")
    y = q.w4a4_linear_static(qa, pw, s, to_dev_bf16(bias_b), 0, workspace=ws)
    torch.cuda.synchronize()
    rows = np.linspace(0, L.M - 1, 96).astype(np.int64)
    a_ref = oracle.quantize_act_static(np.ascontiguousarray(xb[rows]), s, 16)
    wq_ref, sw_ref = oracle.quantize_weight_per_channel(wb)
    y64, S = oracle.linear_static_f64(a_ref, s, wq_ref, sw_ref, bias_b, 0)
    _check(y[torch.from_numpy(rows).cuda()], y64, S, L.K, 0)
