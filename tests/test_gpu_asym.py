"""GPU parity of the asymmetric mode (Eq. 1's zero point, repaired to 255
signed levels over each group's range including 0; reading R9): the
quantizer's codes, flags, scales and zero points bit for bit, the weight
group sums bit for bit, and quartz_w4a4_linear_asym (P_g - z W_g per group,
one correction MFMA per tile) within the output tolerance of tests/helpers.py,
with and without the stream-K workspace."""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import bf16_bits_to_f64, to_dev_bf16, to_host_u16, y_tolerance

pytestmark = pytest.mark.gpu


def _q():
    import paper_2509_26436_amd as q
    return q


def _check_act(qa, ref):
    np.testing.assert_array_equal(to_host_u16(qa.scales), ref.abi_scales)
    np.testing.assert_array_equal(qa.zeros.cpu().numpy(), ref.abi_zeros)
    np.testing.assert_array_equal(qa.flags.cpu().numpy(), ref.abi_flags)
    np.testing.assert_array_equal(qa.codes.cpu().numpy(), ref.codes)


@pytest.mark.parametrize("gs", [8, 16, 32, 64])
@pytest.mark.parametrize("cfg,layer,M", [(1, 0, 200), (2, 3, 77), (5, 0, 129), (3, 3, 1)])
def test_asym_quantizer_bit_exact(cfg, layer, M, gs):
    import torch
    q = _q()
    xb = W.make_x(cfg, layer, rows=M)
    print(f"asym quantize cfg={cfg} layer={layer} M={M} gs={gs}", flush=True)
    qa = q.quantize_act(to_dev_bf16(xb), gs, mode=q.MODE_ASYMMETRIC)
    torch.cuda.synchronize()
    _check_act(qa, oracle.quantize_act_asym(xb, gs))


def test_asym_quantizer_edge_groups():
    """All-positive, all-negative, constant, zero and tiny groups, strided rows."""
    import torch
    q = _q()
    g = np.random.Generator(np.random.PCG64(3))
    K = 448
    rows = []
    rows.append(np.abs(g.laplace(0, 0.1, K)))                 # one-signed, lo = 0
    rows.append(-np.abs(g.laplace(0, 0.1, K)))                # one-signed, hi = 0
    rows.append(np.full(K, 0.37))                             # constant
    rows.append(np.zeros(K))                                  # zero groups: s = 0
    rows.append(g.normal(0, 1e-6, K))                         # subnormal scales
    rows.append(g.normal(0, 3e4, K))                          # large values
    xb = W.to_bf16_bits(np.stack(rows))
    pad = np.zeros((xb.shape[0], K + 24), np.uint16)
    pad[:, :K] = xb
    x = to_dev_bf16(pad)[:, :K]
    qa = q.quantize_act(x, 16, mode=q.MODE_ASYMMETRIC)
    torch.cuda.synchronize()
    _check_act(qa, oracle.quantize_act_asym(xb, 16))


@pytest.mark.parametrize("N,K", [(136, 192), (1, 64), (1152, 4608)])
def test_weight_group_sums_bit_exact(N, K):
    import torch
    q = _q()
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N + K)).normal(0, 0.02, (N, K)))
    pw = q.pack_weight(to_dev_bf16(wb))
    sums = q.weight_group_sums(pw)
    torch.cuda.synchronize()
    wq, _ = oracle.quantize_weight(wb)
    np.testing.assert_array_equal(sums.cpu().numpy(), oracle.weight_group_sums(wq).T)


CASES = [
    # (cfg, layer, M, N, gs, epilogue, bias, workspace)
    (1, 0, 200, 136, 16, 0, True, False),
    (2, 3, 160, 448, 16, 0, True, True),      # post-GELU input, split along K
    (3, 0, 300, 200, 8, 1, False, True),      # ragged, GELU, no bias
    (5, 0, 257, 320, 64, 1, True, False),     # post-SiLU im2col input
    (3, 3, 64, 129, 32, 0, True, True),       # K = 12288
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"cfg{c[0]}l{c[1]}-{c[2]}x{c[3]}-gs{c[4]}"
                         f"{'-ws' if c[7] else ''}")
def test_asym_linear_parity(case):
    import torch
    q = _q()
    cfg, layer, M, N, gs, epi, with_bias, use_ws = case
    K = W.CONFIGS[cfg].layers[layer].K
    print(f"asym linear cfg={cfg} layer={layer} M={M} N={N} K={K} gs={gs} ws={use_ws}", flush=True)
    xb = W.make_x(cfg, layer, rows=M)
    wb = W.make_w(cfg, layer, rows=N)
    bias_b = W.make_bias(cfg, layer, cols=N) if with_bias else None
    qa = q.quantize_act(to_dev_bf16(xb), gs, mode=q.MODE_ASYMMETRIC)
    pw = q.pack_weight(to_dev_bf16(wb))
    sums = q.weight_group_sums(pw)
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    bias = None if bias_b is None else to_dev_bf16(bias_b)
    y = q.w4a4_linear_asym(qa, pw, sums, bias, epi, workspace=ws)
    torch.cuda.synchronize()
    a_ref = oracle.quantize_act_asym(xb, gs)
    wq, sw = oracle.quantize_weight(wb)
    y64, S = oracle.linear_asym_f64(a_ref, wq, sw, bias_b, epi)
    err = np.abs(bf16_bits_to_f64(to_host_u16(y)) - y64)
    tol = y_tolerance(y64, S, K, gelu=(epi == 1))
    bad = err > tol
    assert not bad.any(), f"{bad.sum()} outputs out of tolerance; worst excess {(err - tol).max():.3e}"


def _sample(n: int, count: int, seed: int, tile: int) -> np.ndarray:
    """Sorted distinct indices < n: both ends, both sides of the first and of
    the last tile boundary, plus seeded random ones."""
    fixed = {0, 1, n - 1, n - 2, tile - 1, tile, n // tile * tile - 1, n // tile * tile}
    rng = np.random.Generator(np.random.PCG64(seed))
    rest = rng.choice(n, size=min(n, count), replace=False)
    return np.array(sorted({i for i in fixed if 0 <= i < n} | set(int(i) for i in rest)), np.int64)


@pytest.mark.parametrize("layer", [0, 3], ids=["qkv", "fc2"])
def test_asym_full_size_flux(layer):
    """A FLUX block layer at full size through the workspace entry point, the
    launch the bench times (qkv splits its last round along K, fc2 every tile):
    the quantizer bit for bit and the outputs within tolerance on a sampled
    grid of rows (tiles of 128) and columns (tiles of 256)."""
    import torch
    q = _q()
    L = W.CONFIGS[3].layers[layer]
    gs = 16
    print(f"asym full size {L.name} M={L.M} K={L.K} N={L.N}", flush=True)
    xb, wb, bias_b = W.make_x(3, layer), W.make_w(3, layer), W.make_bias(3, layer)
    qa = q.quantize_act(to_dev_bf16(xb), gs, mode=q.MODE_ASYMMETRIC)
    pw = q.pack_weight(to_dev_bf16(wb))
    sums = q.weight_group_sums(pw)
    ws = q.gemm_workspace(L.M, L.N, L.K, "cuda")
    y = q.w4a4_linear_asym(qa, pw, sums, to_dev_bf16(bias_b), L.epilogue, workspace=ws)
    torch.cuda.synchronize()
    rows = _sample(L.M, 32, 700 + layer, 128)
    cols = _sample(L.N, 40, 800 + layer, 256)
    a_ref = oracle.quantize_act_asym(xb[rows], gs)
    r = rows.tolist()
    np.testing.assert_array_equal(qa.codes[:, r, :].cpu().numpy(), a_ref.codes)
    np.testing.assert_array_equal(qa.flags[:, r, :].cpu().numpy(), a_ref.abi_flags)
    np.testing.assert_array_equal(to_host_u16(qa.scales[:, r]), a_ref.abi_scales)
    np.testing.assert_array_equal(qa.zeros[:, r].cpu().numpy(), a_ref.abi_zeros)
    wq, sw = oracle.quantize_weight(wb[cols])
    y64, S = oracle.linear_asym_f64(a_ref, wq, sw, bias_b[cols], L.epilogue)
    got = bf16_bits_to_f64(to_host_u16(y[r][:, cols.tolist()].contiguous()))
    err = np.abs(got - y64)
    tol = y_tolerance(y64, S, L.K, gelu=(L.epilogue == 1))
    bad = err > tol
    assert not bad.any(), f"{bad.sum()} of {bad.size} sampled outputs out of tolerance; worst excess {(err - tol).max():.3e}"
