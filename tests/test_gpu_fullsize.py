"""GPU parity at the full layer sizes of every workload, through the same entry
points and launch configuration that bench.py times.

The GPU processes whole layers (all M rows, all N columns, all K); the CPU
oracle recomputes a sample that spans the first and the ragged last tiles and
random interior rows / columns:
  - activation codes, flags and scales of the sampled rows: bit-exact
    (quantization is row-local, so the oracle on those rows alone is exact);
  - weight codes and scales of the sampled columns: bit-exact;
  - the integer accumulator on the sampled (row, column) grid: bit-exact;
  - the bf16 output on that grid: within the tolerance of tests/helpers.py.
The batched FLUX MLP (fc1 with the GELU epilogue feeding fc2) runs as one
pipeline on the GPU; the sampled rows of fc2's input are overwritten with the
oracle's own fc1 output before fc2 is quantized, so no oracle input comes from
the GPU.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import bf16_bits_to_f64, to_dev_bf16, to_host_u16, y_tolerance

pytestmark = pytest.mark.gpu

GS = 16
FULL_LAYERS = [(c, i) for c in (1, 2, 3, 5) for i in range(len(W.CONFIGS[c].layers))]


def _q():
    import paper_2509_26436_amd as q
    return q


def sample_idx(n: int, count: int, seed: int, tile: int) -> np.ndarray:
    """Sorted distinct indices < n: both ends, both sides of the first tile
    boundaries and of the last (ragged) tile, plus seeded random ones."""
    fixed = {0, 1, n - 1, n - 2, tile - 1, tile, n // tile * tile - 1, n // tile * tile}
    fixed = {i for i in fixed if 0 <= i < n}
    rng = np.random.Generator(np.random.PCG64(seed))
    rest = rng.choice(n, size=min(n, count), replace=False)
    return np.array(sorted(fixed | set(int(i) for i in rest)), dtype=np.int64)


def _check_act_rows(qa, rows, ref):
    codes = qa.codes[:, rows.tolist(), :].cpu().numpy()
    flags = qa.flags[:, rows.tolist(), :].cpu().numpy()
    scales = to_host_u16(qa.scales[:, rows.tolist()])
    np.testing.assert_array_equal(codes, ref.codes)
    np.testing.assert_array_equal(flags, ref.abi_flags)
    np.testing.assert_array_equal(scales, ref.abi_scales)


def _check_weight_cols(q, pw, cols, wb_cols):
    wq = q.unpack_weight(pw)
    got = wq[cols.tolist()].cpu().numpy()
    wq_ref, sw_ref = oracle.quantize_weight(wb_cols)
    np.testing.assert_array_equal(got, wq_ref)
    np.testing.assert_array_equal(to_host_u16(pw.scales[cols.tolist()]), sw_ref)
    return wq_ref, sw_ref


def _check_outputs(y, rows, cols, a_ref, wq_ref, sw_ref, bias_cols, epilogue, K):
    rr, cc = np.meshgrid(np.arange(rows.size), np.arange(cols.size), indexing="ij")
    y64, S = oracle.linear_f64_sampled(a_ref, wq_ref, sw_ref, bias_cols, rr.ravel(), cc.ravel(),
                                       epilogue=epilogue)
    got = y[rows.tolist()][:, cols.tolist()]
    got = bf16_bits_to_f64(to_host_u16(got.contiguous())).ravel()
    tol = y_tolerance(y64, S, K, gelu=(epilogue == 1))
    err = np.abs(got - y64)
    bad = err > tol
    assert not bad.any(), (f"{bad.sum()} of {bad.size} sampled outputs out of tolerance; "
                           f"worst excess {(err - tol).max():.3e}")


@pytest.mark.parametrize("cfg,layer", FULL_LAYERS)
def test_full_size_layer(cfg, layer):
    import torch
    q = _q()
    L = W.CONFIGS[cfg].layers[layer]
    print(f"full-size layer cfg={cfg} {L.name} M={L.M} K={L.K} N={L.N}", flush=True)
    xb = W.make_x(cfg, layer)
    wb = W.make_w(cfg, layer)
    bias = W.make_bias(cfg, layer)
    qa = q.quantize_act(to_dev_bf16(xb), GS)
    pw = q.pack_weight(to_dev_bf16(wb))
    y = q.w4a4_linear(qa, pw, to_dev_bf16(bias), L.epilogue)
    # the workspace entry point, as bench.py times it
    ws = q.gemm_workspace(L.M, L.N, L.K, "cuda")
    y_ws = q.w4a4_linear(qa, pw, to_dev_bf16(bias), L.epilogue, workspace=ws)
    acc = q.w4a4_gemm_i32(qa, pw)
    torch.cuda.synchronize()

    rows = sample_idx(L.M, 40, 7 * cfg + layer, 256)
    cols = sample_idx(L.N, 48, 11 * cfg + layer, 128)
    a_ref = oracle.quantize_act(xb[rows], GS)
    _check_act_rows(qa, rows, a_ref)
    wq_ref, sw_ref = _check_weight_cols(q, pw, cols, wb[cols])
    got_i = acc[rows.tolist()][:, cols.tolist()].cpu().numpy()
    np.testing.assert_array_equal(got_i, oracle.gemm_i32(a_ref, wq_ref))
    _check_outputs(y, rows, cols, a_ref, wq_ref, sw_ref, bias[cols], L.epilogue, L.K)
    _check_outputs(y_ws, rows, cols, a_ref, wq_ref, sw_ref, bias[cols], L.epilogue, L.K)


def test_full_size_flux_mlp_pipeline():
    """Batched FLUX MLP, M = 18432: fc1 (GELU-tanh epilogue) -> quantize -> fc2."""
    import torch
    q = _q()
    cfg = W.CONFIGS[4]
    L1, L2 = cfg.layers
    print(f"pipeline M={L1.M}: fc1 {L1.K}->{L1.N}, fc2 {L2.K}->{L2.N}", flush=True)
    x1 = W.make_x(4, 0)
    w1 = W.make_w(4, 0)
    b1 = W.make_bias(4, 0)
    w2 = W.make_w(4, 1)
    b2 = W.make_bias(4, 1)
    pw1 = q.pack_weight(to_dev_bf16(w1))
    pw2 = q.pack_weight(to_dev_bf16(w2))
    qa1 = q.quantize_act(to_dev_bf16(x1), GS)
    y1 = q.w4a4_linear(qa1, pw1, to_dev_bf16(b1), 1,
                       workspace=q.gemm_workspace(L1.M, L1.N, L1.K, "cuda"))
    torch.cuda.synchronize()

    rows = sample_idx(L1.M, 24, 401, 256)
    cols1 = sample_idx(L1.N, 32, 402, 128)
    cols2 = sample_idx(L2.N, 48, 403, 128)
    a1_ref = oracle.quantize_act(x1[rows], GS)
    _check_act_rows(qa1, rows, a1_ref)
    wq1, sw1 = oracle.quantize_weight(w1)
    _check_outputs(y1, rows, cols1, a1_ref, wq1[cols1], sw1[cols1], b1[cols1], 1, L1.K)

    # the oracle's fc1 output (all N columns of the sampled rows) is fc2's input there
    y1_64, _ = oracle.linear_f64(a1_ref, wq1, sw1, b1, epilogue=1)
    x2_rows = oracle.to_bf16_bits(y1_64)
    y1[rows.tolist()] = to_dev_bf16(x2_rows)
    qa2 = q.quantize_act(y1, GS)
    y2 = q.w4a4_linear(qa2, pw2, to_dev_bf16(b2), 0,
                       workspace=q.gemm_workspace(L2.M, L2.N, L2.K, "cuda"))
    torch.cuda.synchronize()
    a2_ref = oracle.quantize_act(x2_rows, GS)
    _check_act_rows(qa2, rows, a2_ref)
    wq2_ref, sw2_ref = _check_weight_cols(q, pw2, cols2, w2[cols2])
    _check_outputs(y2, rows, cols2, a2_ref, wq2_ref, sw2_ref, b2[cols2], 0, L2.K)
    assert torch.isfinite(y2.float()).all()


@pytest.mark.parametrize("gs", [8, 32, 64])
def test_full_size_flux_qkv_group_sizes(gs):
    """The G_s sweep of the FLUX QKV layer (Table 1's g8 / g16 / g32, plus 64)."""
    import torch
    q = _q()
    L = W.CONFIGS[3].layers[0]
    xb = W.make_x(3, 0)
    wb = W.make_w(3, 0)
    bias = W.make_bias(3, 0)
    qa = q.quantize_act(to_dev_bf16(xb), gs)
    pw = q.pack_weight(to_dev_bf16(wb))
    y = q.w4a4_linear(qa, pw, to_dev_bf16(bias), 0)
    torch.cuda.synchronize()
    rows = sample_idx(L.M, 24, 500 + gs, 256)
    cols = sample_idx(L.N, 32, 600 + gs, 128)
    a_ref = oracle.quantize_act(xb[rows], gs)
    _check_act_rows(qa, rows, a_ref)
    wq_ref, sw_ref = oracle.quantize_weight(wb[cols])
    _check_outputs(y, rows, cols, a_ref, wq_ref, sw_ref, bias[cols], 0, L.K)


def test_max_k():
    """K at the library's limit (2^20, 16384 groups), a few rows."""
    import torch
    q = _q()
    M, N, K = 3, 70, 1 << 20
    xb = W.make_random_x(91, M, K, "t3", 0.05)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(92)).normal(0, 0.02, (N, K)))
    bias = W.to_bf16_bits(np.random.Generator(np.random.PCG64(93)).normal(0, 0.02, N))
    qa = q.quantize_act(to_dev_bf16(xb), GS)
    pw = q.pack_weight(to_dev_bf16(wb))
    y = q.w4a4_linear(qa, pw, to_dev_bf16(bias), 0)
    acc = q.w4a4_gemm_i32(qa, pw)
    torch.cuda.synchronize()
    a_ref = oracle.quantize_act(xb, GS)
    _check_act_rows(qa, np.arange(M), a_ref)
    wq_ref, sw_ref = oracle.quantize_weight(wb)
    np.testing.assert_array_equal(acc.cpu().numpy(), oracle.gemm_i32(a_ref, wq_ref))
    _check_outputs(y, np.arange(M), np.arange(N), a_ref, wq_ref, sw_ref, bias, 0, K)


def test_many_rows():
    """M = 2^20 + 37 rows (4097 row tiles, ragged), one group, small N."""
    import torch
    q = _q()
    M, N, K = (1 << 20) + 37, 72, 64
    xb = W.make_random_x(94, M, K, "laplace", 0.1)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(95)).normal(0, 0.02, (N, K)))
    qa = q.quantize_act(to_dev_bf16(xb), GS)
    pw = q.pack_weight(to_dev_bf16(wb))
    y = q.w4a4_linear(qa, pw, None, 0)
    torch.cuda.synchronize()
    rows = sample_idx(M, 64, 96, 256)
    a_ref = oracle.quantize_act(xb[rows], GS)
    _check_act_rows(qa, rows, a_ref)
    wq_ref, sw_ref = oracle.quantize_weight(wb)
    _check_outputs(y, rows, np.arange(N), a_ref, wq_ref, sw_ref, None, 0, K)
