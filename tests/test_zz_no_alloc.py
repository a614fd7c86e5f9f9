"""quartz_w4a4_linear_noalloc (the layer with the library's device scratch
array in place of a workspace) against quartz_w4a4_linear_ws with a
workspace: the same schedule and split, so the outputs must be bit-identical;
both within the oracle's tolerance on sampled outputs.  Two calls in a row on
the one scratch array, the second with a smaller input, then the first shape
again."""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import bf16_bits_to_f64, to_dev_bf16, to_host_u16, y_tolerance

pytestmark = pytest.mark.gpu

# (M, N, K, G_s, epilogue): both shapes split their tiles along K on 256 workgroups
SHAPES = [(1200, 1000, 3072, 16, 0), (300, 260, 3072, 8, 1)]


def _case(M, N, K, gs, seed):
    import torch
    import paper_2509_26436_amd as q
    xb = W.make_random_x(seed, M, K, "t3", 0.05)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(seed + 1)).normal(0, 0.015, (N, K)))
    bias = W.to_bf16_bits(np.random.Generator(np.random.PCG64(seed + 2)).normal(0, 0.02, N))
    qa = q.quantize_act(to_dev_bf16(xb), gs)
    pw = q.pack_weight(to_dev_bf16(wb))
    return xb, wb, bias, qa, pw, to_dev_bf16(bias)


def _noalloc_vs_ws(M, N, K, gs, epi, seed):
    import torch
    import paper_2509_26436_amd as q
    xb, wb, bias, qa, pw, bias_d = _case(M, N, K, gs, seed)
    sched, _ = q.linear_schedule(M, N, K, torch.cuda.get_device_properties(0).multi_processor_count)
    assert sched["split"] == 1, "the shape must exercise the split path"
    nbytes = q.quartz_w4a4_linear_workspace_bytes(M, N, K)
    assert 0 < nbytes <= q.quartz_w4a4_linear_noalloc_max_bytes()
    ws = q.gemm_workspace(M, N, K, qa.codes.device)
    y_ws = q.w4a4_linear(qa, pw, bias_d, epi, workspace=ws)
    out = torch.full((M, N + 8), -1.0, dtype=torch.bfloat16, device="cuda")
    y_na = q.w4a4_linear_noalloc(qa, pw, out[:, :N], bias_d, epi)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_host_u16(y_na.contiguous()), to_host_u16(y_ws))
    # the columns past N of the strided output are untouched
    assert (out[:, N:] == -1.0).all().item()
    # and within the oracle's tolerance on sampled outputs
    rng = np.random.Generator(np.random.PCG64(seed + 3))
    rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, 24, replace=False)]))
    cols = np.unique(np.concatenate([[0, N - 1], rng.choice(N, 24, replace=False)]))
    a_ref = oracle.quantize_act(xb[rows], gs)
    wq_ref, sw_ref = oracle.quantize_weight(wb[cols])
    rr, cc = np.meshgrid(np.arange(rows.size), np.arange(cols.size), indexing="ij")
    y64, S = oracle.linear_f64_sampled(a_ref, wq_ref, sw_ref, bias[cols], rr.ravel(), cc.ravel(),
                                       epilogue=epi)
    got = bf16_bits_to_f64(to_host_u16(y_na[rows.tolist()][:, cols.tolist()].contiguous())).ravel()
    assert (np.abs(got - y64) <= y_tolerance(y64, S, K, gelu=epi == 1)).all()


def test_noalloc_equals_workspace_entry_point_twice():
    big, small = SHAPES
    _noalloc_vs_ws(*big, seed=71)
    _noalloc_vs_ws(*small, seed=72)      # second call, smaller input, same scratch array
    _noalloc_vs_ws(*big, seed=73)        # and the larger shape again after it
