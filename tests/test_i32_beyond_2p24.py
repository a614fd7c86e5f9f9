"""The exact integer accumulator (quartz_w4a4_gemm_i32) where the sum over K
leaves the range fp32 holds exactly.

Section 4.4's integer MMA accumulates s4 x s4 products exactly in s32.  The
per-group products P_g are exact in any case (|P_g| <= 112 * 7 * 64 < 2^24),
but their sum I = sum_g P_g reaches 784 K, above 2^24 once K > 21398; the
inputs below make |I| > 2^24 with odd low bits, which an fp32 sum of the
groups would round.

Construction (every scale a power of two, so Stage 1 returns the chosen
integers themselves): in the first BIG groups of a row all 64 values equal
+-t (q = 127 -> FLAG 4 -> c = 7, d = 112); in the other groups the first value
is 127 t (the group maximum: its subgroup has FLAG 4, so the small values
beside it truncate to 0) and the rest are q t with q random in [-7, 7], whose
subgroups have FLAG 0 (d = q, odd half of the time).  The weights are 7 u in
the BIG groups and odd multiples of u (a 7 u among them) elsewhere.
"""
import numpy as np
import pytest

import oracle
import workloads as W

K = 32768
BIG = 400
T = 2.0 ** -6          # activation group scale (fp16 of 127 T / 127 = T, normal)
U = 2.0 ** -8          # weight group scale


def make_case(M, N, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    G = K // 64
    sign = np.where(np.arange(M) % 2 == 0, 1.0, -1.0)[:, None]
    x = np.empty((M, K))
    x[:, :BIG * 64] = sign * T
    rest = rng.integers(-7, 8, size=(M, (G - BIG) * 64)).astype(np.float64)
    rest[:, ::64] = 127.0
    x[:, BIG * 64:] = rest * T
    w = np.empty((N, K))
    w[:, :BIG * 64] = 7.0 * U
    odd = rng.choice(np.array([-7, -5, -3, -1, 1, 3, 5, 7], np.float64), size=(N, (G - BIG) * 64))
    odd[:, 1::64] = 7.0
    w[:, BIG * 64:] = odd * U
    return W.to_bf16_bits(x), W.to_bf16_bits(w)


@pytest.mark.parametrize("gs", [8, 16])
def test_case_reaches_the_inexact_range(gs):
    """On the CPU: the oracle's I exceeds 2^24 in magnitude on every output and
    is odd on a good share of them (an fp32 group sum could not hold it), and
    the oracle's Stage 1 returns the integers the construction chose."""
    xb, wb = make_case(8, 16, 7)
    a = oracle.quantize_act(xb, gs)
    wq, _ = oracle.quantize_weight(wb)
    assert (a.q8[:, :BIG * 64] == np.where(np.arange(8) % 2 == 0, 127, -127)[:, None]).all()
    assert (wq[:, :BIG * 64] == 7).all()
    I = oracle.gemm_i32(a, wq).astype(np.int64)
    assert (np.abs(I) > 2 ** 24).all()
    # (the parity of I is that of the row's count of odd FLAG-0 values: the
    # weights there are all odd)
    assert 0.2 < (I % 2 != 0).mean() < 0.8
    # the same sum rounded through fp32 group by group differs
    d = a.decoded().astype(np.int64)
    P = np.einsum("mgk,ngk->mng", d.reshape(8, -1, 64), wq.astype(np.int64).reshape(16, -1, 64))
    f32 = np.zeros((8, 16), np.float32)
    for g in range(P.shape[2]):
        f32 = (f32 + P[:, :, g].astype(np.float32)).astype(np.float32)
    assert (f32.astype(np.int64) != I).any()


@pytest.mark.gpu
@pytest.mark.parametrize("gs", [8, 16])
def test_gemm_i32_exact_beyond_2p24(gs):
    """GPU quantizer, pack and integer accumulator at K = 32768 against the
    oracle, bit for bit (rows and columns span a ragged tile)."""
    import torch
    import paper_2509_26436_amd as q
    from helpers import to_dev_bf16
    M, N = 70, 136
    xb, wb = make_case(M, N, 11 + gs)
    qa = q.quantize_act(to_dev_bf16(xb), gs)
    pw = q.pack_weight(to_dev_bf16(wb))
    acc = q.w4a4_gemm_i32(qa, pw)
    torch.cuda.synchronize()
    a_ref = oracle.quantize_act(xb, gs)
    wq_ref, _ = oracle.quantize_weight(wb)
    ref = oracle.gemm_i32(a_ref, wq_ref)
    assert (np.abs(ref.astype(np.int64)) > 2 ** 24).all()
    np.testing.assert_array_equal(acc.cpu().numpy(), ref)
