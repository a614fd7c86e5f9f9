"""Output bounds of every bf16-output GEMM entry point: the output is a view of
the first M rows (and N columns) of a larger buffer filled with a sentinel;
after the call the sentinel rows and columns must be untouched and the view
must equal the output of the same call into a fresh tensor.  M is chosen so
that the last tile row ends inside a wave's 64 rows (M % 64 != 0), which is
where a store whose row offset escaped the bounds check would land in the
guard rows; with and without the stream-K workspace, bias and GELU, per-group,
static (LDM) and asymmetric modes."""
import numpy as np
import pytest

import workloads as W
from helpers import to_dev_bf16
from test_gpu_parity import _gemm_case

pytestmark = pytest.mark.gpu

GUARD_ROWS = 64
SENTINEL = 5.0


def _q():
    import paper_2509_26436_amd as q
    return q


def _guarded(call, M, N, pad):
    """Runs call(out) on a guarded view and on a fresh tensor; returns both."""
    import torch
    buf = torch.full((M + GUARD_ROWS, N + pad), SENTINEL, dtype=torch.bfloat16, device="cuda")
    call(buf[:M, :N])
    fresh = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    call(fresh)
    torch.cuda.synchronize()
    s = torch.tensor(SENTINEL, dtype=torch.bfloat16).view(torch.int16).item()
    guard_rows = buf[M:].view(torch.int16)
    assert torch.all(guard_rows == s), f"{int((guard_rows != s).sum())} guard-row elements written"
    if pad:
        assert torch.all(buf[:M, N:].view(torch.int16) == s), "pad columns written"
    assert torch.equal(buf[:M, :N].view(torch.int16), fresh.view(torch.int16))


SHAPES = [
    # (M, N, K, gs, epilogue, bias, workspace, pad)
    (200, 136, 192, 16, 0, True, False, 0),
    (37, 64, 128, 8, 1, True, False, 6),
    (1, 128, 64, 64, 0, False, False, 0),
    (257, 129, 1152, 32, 0, True, True, 0),     # two tiles split along K
    (130, 320, 576, 16, 1, False, True, 4),
]


@pytest.mark.parametrize("case", SHAPES, ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}-gs{c[3]}"
                         f"-e{c[4]}{'-ws' if c[6] else ''}")
def test_per_group_output_stays_in_bounds(case):
    q = _q()
    M, N, K, gs, epi, with_bias, use_ws, pad = case
    print(f"bounds per-group M={M} N={N} K={K} gs={gs} epi={epi} ws={use_ws}", flush=True)
    xb = W.make_random_x(M * 3 + N, M, K, "t3", 0.05)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 5 + K)).normal(0, 0.02, (N, K)))
    qa, pw, _, _, _ = _gemm_case(xb, wb, gs)
    bias = to_dev_bf16(W.to_bf16_bits(np.linspace(-0.3, 0.3, N))) if with_bias else None
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    _guarded(lambda out: q.w4a4_linear(qa, pw, bias, epi, out=out, workspace=ws), M, N, pad)


@pytest.mark.parametrize("case", SHAPES, ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}-gs{c[3]}"
                         f"-e{c[4]}{'-ws' if c[6] else ''}")
def test_static_output_stays_in_bounds(case):
    q = _q()
    M, N, K, gs, epi, with_bias, use_ws, pad = case
    print(f"bounds static M={M} N={N} K={K} gs={gs} epi={epi} ws={use_ws}", flush=True)
    xb = W.make_random_x(M * 5 + N, M, K, "laplace", 0.1)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 7 + K)).normal(0, 0.02, (N, K)))
    s = float(np.float32(np.abs(W.bf16_bits_to_f32(xb)).max() / 127.0 * 0.7))
    qa = q.quantize_act_static(to_dev_bf16(xb), s, gs)
    pw = q.pack_weight_per_channel(to_dev_bf16(wb))
    bias = to_dev_bf16(W.to_bf16_bits(np.linspace(-0.3, 0.3, N))) if with_bias else None
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    _guarded(lambda out: q.w4a4_linear_static(qa, pw, s, bias, epi, out=out, workspace=ws),
             M, N, pad)


@pytest.mark.parametrize("case", SHAPES, ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}-gs{c[3]}"
                         f"-e{c[4]}{'-ws' if c[6] else ''}")
def test_asym_output_stays_in_bounds(case):
    q = _q()
    M, N, K, gs, epi, with_bias, use_ws, pad = case
    print(f"bounds asym M={M} N={N} K={K} gs={gs} epi={epi} ws={use_ws}", flush=True)
    xb = W.make_random_x(M * 9 + N, M, K, "laplace", 0.1)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 11 + K)).normal(0, 0.02, (N, K)))
    qa = q.quantize_act(to_dev_bf16(xb), gs, mode=q.MODE_ASYMMETRIC)
    pw = q.pack_weight(to_dev_bf16(wb))
    sums = q.weight_group_sums(pw)
    bias = to_dev_bf16(W.to_bf16_bits(np.linspace(-0.3, 0.3, N))) if with_bias else None
    ws = q.gemm_workspace(M, N, K, "cuda") if use_ws else None
    _guarded(lambda out: q.w4a4_linear_asym(qa, pw, sums, bias, epi, out=out, workspace=ws),
             M, N, pad)
