"""Every output buffer of every entry point with a guard region after it: each
buffer is the first bytes of a larger allocation filled with a byte pattern;
after the call the pattern past the buffer must be intact, and the buffer must
equal what the same call writes into a plain tensor.  Shapes are ragged (rows
and columns that end inside a tile, a team or a panel), so a store that lost
its bounds would land in the guard."""
import ctypes

import numpy as np
import pytest

import workloads as W
from helpers import to_dev_bf16

pytestmark = pytest.mark.gpu

GUARD = 4096
PATTERN = 0xA5


def _q():
    import paper_2509_26436_amd as q
    return q


class Guarded:
    """A device buffer of `nbytes` followed by GUARD pattern bytes."""

    def __init__(self, nbytes):
        import torch
        self.n = nbytes
        self.buf = torch.full((nbytes + GUARD,), PATTERN, dtype=torch.uint8, device="cuda")

    @property
    def ptr(self):
        return ctypes.c_void_p(self.buf.data_ptr())

    def view(self, dtype):
        return self.buf[:self.n].view(dtype)

    def check(self, what):
        import torch
        g = self.buf[self.n:]
        assert torch.all(g == PATTERN), f"{what}: {int((g != PATTERN).sum())} guard bytes written"


def _same(guarded, plain, what):
    import torch
    guarded.check(what)
    a = guarded.view(torch.uint8)
    b = plain.contiguous().view(-1).view(torch.uint8)
    assert torch.equal(a, b), f"{what}: guarded output differs from the plain call"


def _act_sizes(M, K, gs):
    G = K // 64
    return {"codes": G * M * 32, "flags": G * M * (64 // gs), "scales": G * M * 2, "zeros": G * M}


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("gs", [8, 16, 32, 64])
@pytest.mark.parametrize("M,K", [(37, 192), (200, 576), (1, 64)])
def test_quantizer_outputs(M, K, gs, mode):
    import torch
    q = _q()
    print(f"guard quantize_act M={M} K={K} gs={gs} mode={mode}", flush=True)
    x = to_dev_bf16(W.make_random_x(M + K + gs, M, K, "laplace", 0.1))
    ref = q.quantize_act(x, gs, with_zeros=True, mode=mode)
    bufs = {k: Guarded(n) for k, n in _act_sizes(M, K, gs).items()}
    st = q.quartz_quantize_act(q._ptr(x), M, K, x.stride(0), 64, gs, mode, bufs["codes"].ptr,
                               bufs["flags"].ptr, bufs["scales"].ptr, bufs["zeros"].ptr,
                               q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    for k in bufs:
        _same(bufs[k], getattr(ref, k), k)


@pytest.mark.parametrize("gs", [8, 16, 64])
@pytest.mark.parametrize("M,K", [(37, 192), (200, 576)])
def test_static_quantizer_outputs(M, K, gs):
    import torch
    q = _q()
    print(f"guard quantize_act_static M={M} K={K} gs={gs}", flush=True)
    xb = W.make_random_x(M * 3 + K, M, K, "t3", 0.05)
    s = float(np.float32(np.abs(W.bf16_bits_to_f32(xb)).max() / 127.0 * 0.6))
    x = to_dev_bf16(xb)
    ref = q.quantize_act_static(x, s, gs)
    sizes = _act_sizes(M, K, gs)
    codes, flags = Guarded(sizes["codes"]), Guarded(sizes["flags"])
    st = q.quartz_quantize_act_static(q._ptr(x), M, K, x.stride(0), s, gs, codes.ptr, flags.ptr,
                                      q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    _same(codes, ref.codes, "codes")
    _same(flags, ref.flags, "flags")


@pytest.mark.parametrize("N,K", [(136, 192), (1, 64), (129, 1152), (64, 128)])
def test_pack_unpack_and_sums_outputs(N, K):
    import torch
    q = _q()
    print(f"guard pack N={N} K={K}", flush=True)
    w = to_dev_bf16(W.to_bf16_bits(np.random.Generator(np.random.PCG64(N + 3 * K)).normal(0, 0.02, (N, K))))
    ref = q.pack_weight(w)
    nbytes = q.quartz_packed_weight_bytes(N, K, 64)
    packed, scales = Guarded(nbytes), Guarded(N * (K // 64) * 2)
    st = q.quartz_pack_weight(q._ptr(w), N, K, 64, packed.ptr, scales.ptr, q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    _same(packed, ref.data[:nbytes], "w_packed")
    _same(scales, ref.scales, "w_scales")

    ref_pc = q.pack_weight_per_channel(w)
    packed_pc, scales_pc = Guarded(nbytes), Guarded(N * 2)
    st = q.quartz_pack_weight_per_channel(q._ptr(w), N, K, packed_pc.ptr, scales_pc.ptr,
                                          q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    _same(packed_pc, ref_pc.data[:nbytes], "w_packed (per channel)")
    _same(scales_pc, ref_pc.scales, "w_scales (per channel)")

    sums = Guarded((K // 64) * N * 2)
    st = q.quartz_weight_group_sums(q._ptr(ref.data), N, K, 64, sums.ptr, q._stream_handle())
    assert st == q.QUARTZ_OK
    wq = Guarded(N * K)
    st = q.quartz_unpack_weight(q._ptr(ref.data), N, K, 64, wq.ptr, q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    _same(sums, q.weight_group_sums(ref), "weight group sums")
    _same(wq, q.unpack_weight(ref), "unpacked weight")


@pytest.mark.parametrize("M,N,K,gs", [(200, 136, 192, 16), (37, 129, 1152, 8), (1, 64, 64, 64)])
def test_integer_accumulator_output(M, N, K, gs):
    import torch
    q = _q()
    print(f"guard gemm_i32 M={M} N={N} K={K} gs={gs}", flush=True)
    x = to_dev_bf16(W.make_random_x(M * 5 + N, M, K, "t3", 0.05))
    w = to_dev_bf16(W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 9 + K)).normal(0, 0.02, (N, K))))
    qa, pw = q.quantize_act(x, gs), q.pack_weight(w)
    ref = q.w4a4_gemm_i32(qa, pw)
    acc = Guarded(M * N * 4)
    st = q.quartz_w4a4_gemm_i32(q._ptr(qa.codes), q._ptr(qa.flags), q._ptr(pw.data), acc.ptr, M, N,
                                K, 64, gs, q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    _same(acc, ref, "int32 accumulator")


@pytest.mark.parametrize("M,N,K,gs,out_gs,ws", [(200, 128, 192, 16, 16, False),
                                                (37, 192, 576, 8, 32, True),
                                                (257, 64, 1152, 32, 8, True)])
def test_quantizing_linear_outputs(M, N, K, gs, out_gs, ws):
    import torch
    q = _q()
    print(f"guard linear_quantize M={M} N={N} K={K} gs={gs} out_gs={out_gs} ws={ws}", flush=True)
    x = to_dev_bf16(W.make_random_x(M * 13 + N, M, K, "laplace", 0.1))
    w = to_dev_bf16(W.to_bf16_bits(np.random.Generator(np.random.PCG64(N * 17 + K)).normal(0, 0.02, (N, K))))
    bias = to_dev_bf16(W.to_bf16_bits(np.linspace(-0.2, 0.2, N)))
    qa, pw = q.quantize_act(x, gs), q.pack_weight(w)
    work = q.gemm_workspace(M, N, K, "cuda") if ws else None
    ref = q.w4a4_linear_quantize(qa, pw, bias, 1, out_gs, with_zeros=True, workspace=work)
    bufs = {k: Guarded(n) for k, n in _act_sizes(M, N, out_gs).items()}
    nbytes = 0 if work is None else work.numel()
    st = q.quartz_w4a4_linear_quantize(q._ptr(qa.codes), q._ptr(qa.flags), q._ptr(qa.scales), None,
                                       q._ptr(pw.data), q._ptr(bias), M, N, K, 64, gs, 1, out_gs,
                                       q.MODE_SYMMETRIC, bufs["codes"].ptr, bufs["flags"].ptr,
                                       bufs["scales"].ptr, bufs["zeros"].ptr, q._ptr(work), nbytes,
                                       q._stream_handle())
    assert st == q.QUARTZ_OK
    torch.cuda.synchronize()
    for k in bufs:
        _same(bufs[k], getattr(ref, k), k)
