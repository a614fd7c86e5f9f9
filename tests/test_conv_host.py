"""Host-side checks of the implicit 3 x 3 convolution (quartz_w4a4_conv3x3):
the reading that makes it exact (quantizing the feature map once gives, by
tap, the codes, FLAGs and scales of every im2col row, since each 64-group of
an im2col row with C % 64 == 0 is one pixel's 64 channels or zero padding),
checked with the oracle in both settings; the host im2col against a plain
loop; the division by C / 64 the GEMM does with a multiply-high, over its
whole domain; and the entry points' argument validation (no GPU needed)."""
import numpy as np
import pytest

import oracle
import paper_2509_26436_amd as q
import workloads as W

OK, ENULL, ESHAPE, EUNSUP, EALIGN = 0, 1, 2, 3, 4
A = 4096      # a fake, 16-byte aligned address: never dereferenced on these paths


def _fmap(seed, images, H, Wd, C):
    x = np.random.Generator(np.random.PCG64(seed)).laplace(0.0, 0.1, size=(images, H, Wd, C))
    x[..., ::17] *= 25.0
    return W.to_bf16_bits(x)


def _im2col_images(fm):
    return np.concatenate([W.im2col3x3(fm[i]) for i in range(fm.shape[0])], axis=0)


def test_im2col_against_a_plain_loop():
    fm = np.arange(2 * 3 * 4 * 2).reshape(2 * 3, 4, 2)[:3]      # one 3 x 4 map, C = 2
    cols = W.im2col3x3(fm)
    for r in range(12):
        oy, ox = divmod(r, 4)
        for kh in range(3):
            for kw in range(3):
                iy, ix = oy + kh - 1, ox + kw - 1
                want = fm[iy, ix] if 0 <= iy < 3 and 0 <= ix < 4 else np.zeros(2)
                np.testing.assert_array_equal(cols[r, (3 * kh + kw) * 2:(3 * kh + kw + 1) * 2], want)


@pytest.mark.parametrize("H,Wd,C", [(1, 1, 3), (3, 4, 2), (5, 7, 64), (6, 3, 128)])
def test_im2col_against_torch_unfold(H, Wd, C):
    """The host im2col against torch.nn.functional.unfold (kernel 3, padding 1):
    unfold orders K as (c, kh, kw), so its columns are permuted to (kh, kw, c)
    with c fastest, the order the convolution layers use."""
    import torch
    fm = np.random.Generator(np.random.PCG64(1000 + H * Wd * C)).normal(size=(H, Wd, C))
    cols = W.im2col3x3(fm)
    t = torch.from_numpy(np.ascontiguousarray(fm.transpose(2, 0, 1)))[None]      # [1][C][H][W]
    u = torch.nn.functional.unfold(t, kernel_size=3, padding=1)[0]             # [C*9][H*W]
    ref = u.reshape(C, 3, 3, H * Wd).permute(3, 1, 2, 0).reshape(H * Wd, 9 * C).numpy()
    np.testing.assert_array_equal(cols, ref)


def test_im2col_gemm_equals_torch_conv2d():
    """The (kh, kw, c) im2col matrix times the weight [N][9 C] laid out the same
    way equals torch's float64 conv2d (stride 1, padding 1) of the map: the
    convention the implicit GEMM and the oracle's input share is the usual
    convolution, not just the builder's own loop."""
    import torch
    rng = np.random.Generator(np.random.PCG64(1001))
    H, Wd, C, N = 5, 6, 64, 7
    fm = rng.normal(size=(H, Wd, C))
    wt = rng.normal(size=(N, C, 3, 3))                          # torch layout [N][C][kh][kw]
    w_rows = wt.transpose(0, 2, 3, 1).reshape(N, 9 * C)         # [N][(kh, kw, c)]
    y = W.im2col3x3(fm) @ w_rows.T                              # [H*W][N]
    ref = torch.nn.functional.conv2d(torch.from_numpy(np.ascontiguousarray(fm.transpose(2, 0, 1)))[None],
                                     torch.from_numpy(wt), padding=1)[0]       # [N][H][W]
    np.testing.assert_allclose(y, ref.permute(1, 2, 0).reshape(H * Wd, N).numpy(), rtol=1e-12, atol=1e-12)


def _gathered(per_pixel, images, H, Wd, C, zero):
    """Rows of the im2col matrix built from a per-pixel, per-channel-block array
    [C/64][images*H*W][...] by tap, `zero` where the tap leaves the image."""
    cg = C // 64
    rows = images * H * Wd
    out = np.empty((9 * cg, rows) + per_pixel.shape[2:], per_pixel.dtype)
    for m in range(rows):
        img, rem = divmod(m, H * Wd)
        h, w = divmod(rem, Wd)
        for t in range(9):
            hh, ww = h + t // 3 - 1, w + t % 3 - 1
            inside = 0 <= hh < H and 0 <= ww < Wd
            src = (img * H + hh) * Wd + ww
            for cb in range(cg):
                out[t * cg + cb, m] = per_pixel[cb, src] if inside else zero
    return out


@pytest.mark.parametrize("gs", [8, 16, 64])
@pytest.mark.parametrize("images,H,Wd,C", [(1, 5, 7, 64), (2, 3, 4, 128)])
def test_feature_map_codes_are_the_im2col_codes(images, H, Wd, C, gs):
    fm = _fmap(H * Wd + C + gs, images, H, Wd, C)
    a_map = oracle.quantize_act(fm.reshape(-1, C), gs)
    a_col = oracle.quantize_act(_im2col_images(fm), gs)
    np.testing.assert_array_equal(a_col.codes, _gathered(a_map.codes, images, H, Wd, C, 0))
    np.testing.assert_array_equal(a_col.abi_flags, _gathered(a_map.abi_flags, images, H, Wd, C, 0))
    np.testing.assert_array_equal(a_col.abi_scales, _gathered(a_map.abi_scales, images, H, Wd, C, 0))
    s = float(np.float32(np.abs(W.bf16_bits_to_f32(fm)).max() / 127.0 * 0.5))
    st_map = oracle.quantize_act_static(fm.reshape(-1, C), s, gs)
    st_col = oracle.quantize_act_static(_im2col_images(fm), s, gs)
    np.testing.assert_array_equal(st_col.codes, _gathered(st_map.codes, images, H, Wd, C, 0))
    np.testing.assert_array_equal(st_col.abi_flags, _gathered(st_map.abi_flags, images, H, Wd, C, 0))


def test_config5_feature_map_is_the_im2col_source():
    for layer in range(3):
        L = W.CONFIGS[5].layers[layer]
        rows = L.K // 9 // 10
        H = int(round(L.M ** 0.5))
        fm = W.make_feature_map(5, layer, img_rows=rows // H + 2)
        np.testing.assert_array_equal(W.im2col3x3(fm, rows=rows), W.make_x(5, layer, rows=rows))


def test_tap_division_by_multiply_high():
    """g // cg == (g * (floor(2^32 / cg) + 1)) >> 32 for every cg >= 2 with
    9 * 64 * cg <= 2^20 and every group g < 9 cg of such a convolution, and for
    every g < 2^14 at the largest cg."""
    for cg in range(2, (1 << 20) // (9 * 64) + 1):
        magic = (1 << 32) // cg + 1
        g = np.arange(9 * cg, dtype=np.uint64)
        np.testing.assert_array_equal((g * np.uint64(magic)) >> np.uint64(32), g // np.uint64(cg))
    cg = (1 << 20) // (9 * 64)
    g = np.arange(1 << 14, dtype=np.uint64)
    np.testing.assert_array_equal((g * np.uint64((1 << 32) // cg + 1)) >> np.uint64(32), g // np.uint64(cg))


def test_conv_entry_validation():
    if not __import__("os").path.exists(q.library_path()):
        pytest.skip("libquartz.so not built")
    cv = q.quartz_w4a4_conv3x3

    def call(images=1, H=8, Wd=8, C=64, N=8, ldy=8, gs=64, lzs=16, epi=0, codes=A, scales=A, y=A,
             ws=None, wsb=0):
        return cv(codes, A, scales, A, None, y, images, H, Wd, C, N, ldy, gs, lzs, epi, ws, wsb, None)
    assert call(epi=3) == EUNSUP
    assert call(gs=32) == EUNSUP
    assert call(lzs=4) == EUNSUP
    assert call(C=96) == ESHAPE
    assert call(C=0) == ESHAPE
    assert call(H=0) == ESHAPE
    assert call(Wd=-1) == ESHAPE
    assert call(images=-1) == ESHAPE
    assert call(images=1, H=1 << 13, Wd=1 << 13) == ESHAPE          # 2^26 pixels
    assert call(images=4, H=1 << 12, Wd=1 << 12) == ESHAPE
    assert call(C=64 * 1821) == ESHAPE                               # 9 C > 2^20
    assert call(ldy=4) == ESHAPE
    assert call(codes=None) == ENULL
    assert call(scales=None) == ENULL
    assert call(y=None) == ENULL
    assert call(y=A + 2) == EALIGN
    assert call(scales=A + 2) == EALIGN
    assert call(ws=A + 4, wsb=1 << 20) == EALIGN
    assert call(images=0) == OK
    assert call(N=0) == OK
    cs = q.quartz_w4a4_conv3x3_static

    def scall(scale=0.01, C=64, y=A, images=1):
        return cs(A, A, scale, A, None, y, images, 8, 8, C, 8, 8, 16, 0, None, 0, None)
    assert scall(scale=float("inf")) == EUNSUP
    assert scall(scale=float("nan")) == EUNSUP
    assert scall(C=32) == ESHAPE
    assert scall(y=None) == ENULL
    assert scall(images=0) == OK
