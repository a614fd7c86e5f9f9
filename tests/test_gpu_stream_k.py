"""GPU parity of the workspace (stream-K) entry point quartz_w4a4_linear_ws.

Shapes are chosen so that, on a device with 256 compute units, the schedule
splits tiles along K: fewer tiles than workgroups (tiles shared by up to eight
workgroups), a ragged number of rounds, every LZS subgroup size, GELU, no
bias and a strided output.  Every output is compared with the oracle within
the tolerance of tests/helpers.py; repeated calls on one workspace must give
bit-identical outputs (the counters are reset, the summation order is fixed);
garbage in the slot part of the workspace must not matter.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import bf16_bits_to_f64, to_dev_bf16, to_host_u16, y_tolerance
from test_gpu_parity import _gemm_case

pytestmark = pytest.mark.gpu


def _q():
    import paper_2509_26436_amd as q
    return q


def _ws_linear(qa, pw, bias_b, epi, ws, ldy_pad=0):
    import torch
    q = _q()
    M, N = qa.M, pw.N
    bias = None if bias_b is None else to_dev_bf16(bias_b)
    if ldy_pad:
        ybuf = torch.full((M, N + ldy_pad), 7.0, dtype=torch.bfloat16, device="cuda")
        q.w4a4_linear(qa, pw, bias, epi, out=ybuf[:, :N], workspace=ws)
        torch.cuda.synchronize()
        assert torch.all(ybuf[:, N:] == 7.0)
        return ybuf[:, :N].contiguous()
    y = q.w4a4_linear(qa, pw, bias, epi, workspace=ws)
    torch.cuda.synchronize()
    return y


def _check(y, a_ref, wq_ref, sw_ref, bias_b, epi, K):
    y64, S = oracle.linear_f64(a_ref, wq_ref, sw_ref, bias_b, epilogue=epi)
    err = np.abs(bf16_bits_to_f64(to_host_u16(y)) - y64)
    tol = y_tolerance(y64, S, K, gelu=(epi == 1))
    bad = err > tol
    assert not bad.any(), (f"{bad.sum()} outputs out of tolerance; worst excess "
                           f"{(err - tol).max():.3e}")


def _schedule_of(M, N, K):
    import torch
    q = _q()
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    return q.linear_schedule(M, N, K, blocks)[0]


CASES = [
    # (cfg, layer, M, N, gs, epilogue, bias, ldy_pad); tiles of 128 x 256
    (2, 3, 160, 448, 16, 0, True, 0),      # 4 tiles x 72 groups over 18 workgroups
    (2, 3, 70, 130, 16, 1, False, 0),      # 1 tile x 72 groups over 4 workgroups, GELU, no bias
    (3, 0, 300, 200, 8, 0, True, 6),       # ragged rows and columns, strided output
    (3, 3, 257, 129, 32, 0, True, 0),      # K = 12288: 3 tiles x 192 groups
    (5, 0, 513, 320, 64, 1, True, 0),      # 10 tiles, GELU
    (2, 3, 64, 1152, 16, 0, True, 0),      # one tile row, 5 tiles x 72 groups
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"cfg{c[0]}l{c[1]}-{c[2]}x{c[3]}-gs{c[4]}")
def test_ws_linear_parity(case):
    import torch
    q = _q()
    cfg, layer, M, N, gs, epi, with_bias, ldy_pad = case
    L = W.CONFIGS[cfg].layers[layer]
    K = L.K
    print(f"stream-K parity cfg={cfg} layer={layer} M={M} N={N} K={K} gs={gs}", flush=True)
    sched = _schedule_of(M, N, K)
    assert sched["split"] == 1, sched
    xb = W.make_x(cfg, layer, rows=M)
    wb = W.make_w(cfg, layer, rows=N)
    bias = W.make_bias(cfg, layer, cols=N) if with_bias else None
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, gs)
    ws = q.gemm_workspace(M, N, K, "cuda")
    assert ws is not None
    y1 = _ws_linear(qa, pw, bias, epi, ws, ldy_pad)
    _check(y1, a_ref, wq_ref, sw_ref, bias, epi, K)
    # the counters were reset: a second call on the same workspace gives the same bits
    y2 = _ws_linear(qa, pw, bias, epi, ws, ldy_pad)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_ws_slot_contents_do_not_matter():
    """Only the counter part must start at zero: fill the slots with 0xFF bytes
    (NaN floats) and the result is unchanged."""
    import torch
    q = _q()
    M, N, K = 160, 448, 4608
    xb = W.make_x(2, 3, rows=M)
    wb = W.make_w(2, 3, rows=N)
    bias = W.make_bias(2, 3, cols=N)
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, 16)
    ws = q.gemm_workspace(M, N, K, "cuda")
    y1 = _ws_linear(qa, pw, bias, 0, ws)
    sched = _schedule_of(M, N, K)
    counter_bytes = -(-sched["sk_tiles"] * 8 * 4 // 256) * 256
    ws[counter_bytes:] = 0xFF
    y2 = _ws_linear(qa, pw, bias, 0, ws)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    _check(y2, a_ref, wq_ref, sw_ref, bias, 0, K)


def test_ws_matches_plain_entry_point_within_order():
    """The workspace path and the whole-tile path differ only in the fp32 order
    of the group sum: both within tolerance, and within a few bf16 ulps."""
    q = _q()
    M, N = 300, 200
    L = W.CONFIGS[3].layers[3]
    xb = W.make_x(3, 3, rows=M)
    wb = W.make_w(3, 3, rows=N)
    bias = W.make_bias(3, 3, cols=N)
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, 16)
    y_plain = q.w4a4_linear(qa, pw, to_dev_bf16(bias), 0)
    y_ws = _ws_linear(qa, pw, bias, 0, q.gemm_workspace(M, N, L.K, "cuda"))
    _check(y_plain, a_ref, wq_ref, sw_ref, bias, 0, L.K)
    _check(y_ws, a_ref, wq_ref, sw_ref, bias, 0, L.K)


def test_ws_null_and_too_small():
    import torch
    q = _q()
    M, N, K = 160, 448, 4608
    xb = W.make_x(2, 3, rows=M)
    wb = W.make_w(2, 3, rows=N)
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, 16)
    need = q.quartz_w4a4_linear_workspace_bytes(M, N, K)
    assert need > 0
    small = torch.zeros(need - 256, dtype=torch.uint8, device="cuda")
    y = torch.full((M, N), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(q.QuartzError) as e:
        q.w4a4_linear(qa, pw, None, 0, out=y, workspace=small)
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert torch.all(y == 3.0)                       # nothing launched
    # NULL workspace through the _ws entry point: the whole-tile path
    import ctypes
    st = q.quartz_w4a4_linear_ws(
        ctypes.c_void_p(qa.codes.data_ptr()), ctypes.c_void_p(qa.flags.data_ptr()),
        ctypes.c_void_p(qa.scales.data_ptr()), None, ctypes.c_void_p(pw.data.data_ptr()), None,
        ctypes.c_void_p(y.data_ptr()), M, N, K, N, 64, 16, 0, None, 0,
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0
    torch.cuda.synchronize()
    _check(y, a_ref, wq_ref, sw_ref, None, 0, K)
