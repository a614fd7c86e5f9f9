"""The C-ABI library loads, exports every symbol include/quartz.h declares,
and rejects invalid arguments on the host before launching anything (these
calls never reach the GPU, so they run without one)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2509_26436_amd as q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "quartz.h")

OK, ENULL, ESHAPE, EUNSUP, EALIGN = 0, 1, 2, 3, 4
A = 4096      # a fake, 16-byte aligned address: never dereferenced on these paths


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(quartz_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(q.library_path()):
        pytest.skip("libquartz.so not built")
    return q.load()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("quartz_quantize_act", "quartz_pack_weight", "quartz_w4a4_linear"):
        assert n in names
    assert set(names) == set(q.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", q.library_path()],
                         capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_status_strings(lib):
    for s in range(6):
        assert len(q.quartz_status_string(s)) > 0
    assert q.quartz_status_string(99) == "unknown status"


def test_packed_weight_bytes(lib):
    # panels of 64 columns, per (panel, group) 64 * 32 code bytes + 64 fp16 scales
    assert q.quartz_packed_weight_bytes(320, 2880, 64) == 5 * 45 * 2176
    assert q.quartz_packed_weight_bytes(1, 64, 64) == 2176
    assert q.quartz_packed_weight_bytes(64, 100, 64) == 0
    assert q.quartz_packed_weight_bytes(64, 64, 32) == 0


def test_quantize_validation(lib):
    f = q.quartz_quantize_act
    assert f(A, 4, 128, 128, 32, 16, 0, A, A, A, None, None) == EUNSUP
    assert f(A, 4, 128, 128, 64, 12, 0, A, A, A, None, None) == EUNSUP
    assert f(A, 4, 128, 128, 64, 16, 5, A, A, A, None, None) == EUNSUP
    assert f(A, 4, 100, 100, 64, 16, 0, A, A, A, None, None) == ESHAPE
    assert f(A, -1, 128, 128, 64, 16, 0, A, A, A, None, None) == ESHAPE
    assert f(A, 4, 128, 64, 64, 16, 0, A, A, A, None, None) == ESHAPE
    assert f(None, 4, 128, 128, 64, 16, 0, A, A, A, None, None) == ENULL
    assert f(A, 4, 128, 128, 64, 16, 0, None, A, A, None, None) == ENULL
    assert f(A + 2, 4, 128, 128, 64, 16, 0, A, A, A, None, None) == EALIGN
    assert f(A, 4, 128, 132, 64, 16, 0, A, A, A, None, None) == EALIGN
    assert f(A, 4, 128, 128, 64, 16, 0, A, A, A + 8, None, None) == EALIGN
    # nothing to do: OK without a launch (null pointers are fine then)
    assert f(None, 0, 128, 128, 64, 16, 0, None, None, None, None, None) == OK
    # size limits: K <= 2^20, rows * K/64 <= 2^28
    K = 1 << 21
    assert f(A, 1, K, K, 64, 16, 0, A, A, A, None, None) == ESHAPE
    assert f(A, (1 << 24) + 1, 1024, 1024, 64, 16, 0, A, A, A, None, None) == ESHAPE


def test_pack_validation(lib):
    f = q.quartz_pack_weight
    assert f(A, 8, 128, 16, A, None, None) == EUNSUP
    assert f(A, 8, 96, 64, A, None, None) == ESHAPE
    assert f(None, 8, 128, 64, A, None, None) == ENULL
    assert f(A, 8, 128, 64, A + 4, None, None) == EALIGN
    assert f(None, 0, 128, 64, None, None, None) == OK
    assert f(A, (1 << 24) + 1, 1024, 64, A, None, None) == ESHAPE
    assert f(A, 1, 1 << 21, 64, A, None, None) == ESHAPE


def test_linear_validation(lib):
    f = q.quartz_w4a4_linear
    args = dict(codes=A, flags=A, scales=A, zeros=None, w=A, bias=None, y=A)

    def call(M=8, N=8, K=128, ldy=8, gs=64, lzs=16, epi=0, **over):
        a = dict(args, **over)
        return f(a["codes"], a["flags"], a["scales"], a["zeros"], a["w"], a["bias"], a["y"],
                 M, N, K, ldy, gs, lzs, epi, None)
    assert call(gs=128) == EUNSUP
    assert call(lzs=4) == EUNSUP
    assert call(epi=7) == EUNSUP
    assert call(K=96) == ESHAPE
    assert call(K=0) == ESHAPE
    assert call(ldy=4) == ESHAPE
    assert call(M=-3) == ESHAPE
    assert call(codes=None) == ENULL
    assert call(y=None) == ENULL
    assert call(w=A + 1) == EALIGN
    assert call(bias=A + 2) == EALIGN
    assert call(M=0) == OK
    assert call(N=0) == OK
    assert call(K=1 << 21) == ESHAPE
    # more than 2^31 - 1 output tiles of 256 x 128
    assert call(M=1 << 28, N=1 << 28, ldy=1 << 28, K=64) == ESHAPE
    assert call(N=(1 << 24) + 1, ldy=(1 << 24) + 1, K=1024) == ESHAPE


def test_linear_quantize_validation(lib):
    f = q.quartz_w4a4_linear_quantize
    args = dict(codes=A, flags=A, scales=A, zeros=None, w=A, bias=None,
                oc=A, of=A, os=A, oz=None, ws=None)

    def call(M=8, N=64, K=128, gs=64, lzs=16, epi=0, olzs=16, omode=0, wsb=0, **over):
        a = dict(args, **over)
        return f(a["codes"], a["flags"], a["scales"], a["zeros"], a["w"], a["bias"], M, N, K,
                 gs, lzs, epi, olzs, omode, a["oc"], a["of"], a["os"], a["oz"], a["ws"], wsb, None)
    assert call(olzs=4) == EUNSUP
    assert call(olzs=128) == EUNSUP
    assert call(omode=1) == EUNSUP
    assert call(gs=32) == EUNSUP
    assert call(epi=3) == EUNSUP
    assert call(N=96) == ESHAPE          # the output is the next layer's K: N % 64 == 0
    assert call(N=32) == ESHAPE
    assert call(K=100) == ESHAPE
    assert call(M=-1) == ESHAPE
    assert call(oc=None) == ENULL
    assert call(of=None) == ENULL
    assert call(os=None) == ENULL
    assert call(scales=None) == ENULL
    assert call(oc=A + 4) == EALIGN
    assert call(oz=A + 8) == EALIGN
    assert call(ws=A + 2, wsb=1 << 20) == EALIGN
    assert call(M=0) == OK
    assert call(N=0) == OK


def test_ldm_entry_validation(lib):
    qs = q.quartz_quantize_act_static
    assert qs(A, 8, 128, 128, 0.0, 16, A, A, None) == EUNSUP
    assert qs(A, 8, 128, 128, -1.0, 16, A, A, None) == EUNSUP
    assert qs(A, 8, 128, 128, float("inf"), 16, A, A, None) == EUNSUP
    assert qs(A, 8, 128, 128, float("nan"), 16, A, A, None) == EUNSUP
    assert qs(A, 8, 128, 128, 1e-40, 16, A, A, None) == EUNSUP      # subnormal: 1/s overflows
    assert qs(A, 8, 128, 128, 0.01, 12, A, A, None) == EUNSUP
    assert qs(A, 8, 100, 128, 0.01, 16, A, A, None) == ESHAPE
    assert qs(A, 8, 128, 64, 0.01, 16, A, A, None) == ESHAPE
    assert qs(A, 8, 128, 132, 0.01, 16, A, A, None) == EALIGN
    assert qs(A, 0, 128, 128, 0.01, 16, A, A, None) == OK
    assert qs(None, 8, 128, 128, 0.01, 16, A, A, None) == ENULL
    assert qs(A, 8, 128, 128, 0.01, 16, A, None, None) == ENULL
    assert qs(A, 8, 128, 128, 0.01, 16, A + 2, A, None) == EALIGN
    pc = q.quartz_pack_weight_per_channel
    assert pc(A, 8, 100, A, None, None) == ESHAPE
    assert pc(A, 0, 128, A, None, None) == OK
    assert pc(None, 8, 128, A, None, None) == ENULL
    assert pc(A, 8, 128, A + 8, None, None) == EALIGN
    assert pc(A, 8, 128, A, A + 2, None) == EALIGN
    ls = q.quartz_w4a4_linear_static

    def call(M=8, N=8, K=128, ldy=8, lzs=16, epi=0, scale=0.01, y=A, codes=A, ws=None, wsb=0):
        return ls(codes, A, scale, A, None, y, M, N, K, ldy, lzs, epi, ws, wsb, None)
    assert call(epi=2) == EUNSUP
    assert call(scale=float("inf")) == EUNSUP
    assert call(lzs=5) == EUNSUP
    assert call(K=96) == ESHAPE
    assert call(ldy=4) == ESHAPE
    assert call(codes=None) == ENULL
    assert call(y=None) == ENULL
    assert call(y=A + 4) == EALIGN
    assert call(ws=A + 4, wsb=1 << 20) == EALIGN
    assert call(M=0) == OK
    assert call(N=0) == OK


def test_asym_entry_validation(lib):
    qa = q.quartz_quantize_act
    assert qa(A, 8, 128, 128, 64, 16, 2, A, A, A, A, None) == EUNSUP      # unknown mode
    assert qa(A, 8, 128, 128, 64, 16, 1, A, A, A, None, None) == ENULL    # asym needs zeros
    assert qa(A, 8, 128, 128, 64, 16, 1, A, A, A, A + 2, None) == EALIGN
    assert qa(A, 0, 128, 128, 64, 16, 1, A, A, A, None, None) == OK
    ws = q.quartz_weight_group_sums
    assert ws(A, 8, 128, 32, A, None) == EUNSUP
    assert ws(A, 8, 100, 64, A, None) == ESHAPE
    assert ws(None, 8, 128, 64, A, None) == ENULL
    assert ws(A, 8, 128, 64, None, None) == ENULL
    assert ws(A, 8, 128, 64, A + 2, None) == EALIGN
    assert ws(A, 0, 128, 64, A, None) == OK
    la = q.quartz_w4a4_linear_asym

    def call(M=8, N=8, K=128, ldy=8, gs=64, lzs=16, epi=0, zeros=A, sums=A, y=A, wsp=None, wsb=0):
        return la(A, A, A, zeros, A, sums, None, y, M, N, K, ldy, gs, lzs, epi, wsp, wsb, None)
    assert call(epi=4) == EUNSUP
    assert call(gs=16) == EUNSUP
    assert call(K=96) == ESHAPE
    assert call(ldy=4) == ESHAPE
    assert call(zeros=None) == ENULL
    assert call(sums=None) == ENULL
    assert call(y=None) == ENULL
    assert call(sums=A + 2) == EALIGN
    assert call(wsp=A + 4, wsb=1 << 20) == EALIGN
    assert call(M=0) == OK


def test_debug_entry_validation(lib):
    assert q.quartz_unpack_weight(A, 8, 100, 64, A, None) == ESHAPE
    assert q.quartz_unpack_weight(None, 8, 128, 64, A, None) == ENULL
    assert q.quartz_w4a4_gemm_i32(A, A, A, None, 8, 8, 128, 64, 16, None) == ENULL
    assert q.quartz_w4a4_gemm_i32(A, A, A, A, 8, 8, 128, 64, 5, None) == EUNSUP
    assert q.quartz_w4a4_gemm_i32(A, A, A, A, 0, 8, 128, 64, 16, None) == OK


def test_product_path_does_not_touch_the_oracle():
    pkg = os.path.join(ROOT, "paper_2509_26436_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in text.lower(), fn


def test_layers_reject_activations_of_another_mode():
    """The tensor helpers refuse codes of a quantizer mode the layer does not
    decode (asymmetric codes into the symmetric layer would drop their zero
    points silently); checked before anything reaches the library."""
    import torch
    G, M, K = 2, 4, 128
    def act(mode):
        return q.QuantizedAct(codes=torch.zeros((G, M, 32), dtype=torch.uint8),
                              flags=torch.zeros((G, M, 4), dtype=torch.uint8),
                              scales=torch.zeros((G, M), dtype=torch.int16),
                              zeros=torch.zeros((G, M), dtype=torch.int8),
                              M=M, K=K, lzs_group=16, mode=mode)
    w = q.PackedWeight(data=torch.zeros(8, dtype=torch.uint8), scales=None, N=64, K=K)
    calls = {
        q.MODE_SYMMETRIC: [lambda a: q.w4a4_linear(a, w), lambda a: q.w4a4_linear_quantize(a, w)],
        q.MODE_ASYMMETRIC: [lambda a: q.w4a4_linear_asym(a, w, None)],
        q.MODE_STATIC: [lambda a: q.w4a4_linear_static(a, w, 1.0)],
    }
    for want, fns in calls.items():
        for other in calls:
            if other == want:
                continue
            for fn in fns:
                with pytest.raises(ValueError, match="mode"):
                    fn(act(other))


def test_attention_entry_validation(lib):
    EWS = 6
    vt = q.quartz_quantize_vt
    assert vt(A, 2, 128, 128, 128, 12, A, A, A, None) == EUNSUP
    assert vt(A, 2, 100, 128, 128, 16, A, A, A, None) == ESHAPE       # L % 64
    assert vt(A, 2, 128, 96, 128, 16, A, A, A, None) == ESHAPE        # d % 64
    assert vt(A, 2, 128, 128, 64, 16, A, A, A, None) == ESHAPE        # ldv < d
    assert vt(A, 2, 128, 128, 132, 16, A, A, A, None) == EALIGN       # ldv % 8
    assert vt(A, 0, 128, 128, 128, 16, A, A, A, None) == OK
    assert vt(None, 2, 128, 128, 128, 16, A, A, A, None) == ENULL
    assert vt(A + 2, 2, 128, 128, 128, 16, A, A, A, None) == EALIGN
    sm = q.quartz_softmax_quantize
    assert sm(A, 8, 128, 128, 5, A, A, A, None) == EUNSUP
    assert sm(A, 8, 100, 128, 16, A, A, A, None) == ESHAPE            # N % 64
    assert sm(A, 8, 128, 64, 16, A, A, A, None) == ESHAPE             # lds < N
    assert sm(A, 8, 128, 130, 16, A, A, A, None) == EALIGN            # lds % 4
    assert sm(A, 0, 128, 128, 16, A, A, A, None) == OK
    assert sm(None, 8, 128, 128, 16, A, A, A, None) == ENULL
    assert sm(A + 4, 8, 128, 128, 16, A, A, A, None) == EALIGN
    sc = q.quartz_attn_scores

    def scores(q_plane=256, q_row0=0, Lq=128, Lk=128, d=128, gs=16, scale=0.1, s=A, lds=128):
        return sc(A, A, A, q_plane, q_row0, A, A, A, 256, 0, Lq, Lk, d, gs, scale, s, lds, None)
    assert scores(scale=float("inf")) == EUNSUP
    assert scores(gs=3) == EUNSUP
    assert scores(d=96) == ESHAPE
    assert scores(q_row0=200) == ESHAPE                                # rows past the plane
    assert scores(lds=64) == ESHAPE
    assert scores(Lq=0) == OK
    assert scores(s=None) == ENULL
    assert scores(s=A + 4) == EALIGN
    pv = q.quartz_attn_pv

    def pvc(vt_plane=256, vt_row0=0, Lq=128, Lk=128, d=128, o=A, ldo=128, ws=None, wsb=0):
        return pv(A, A, A, A, A, A, vt_plane, vt_row0, Lq, Lk, d, 16, o, ldo, ws, wsb, None)
    assert pvc(Lk=100) == ESHAPE
    assert pvc(vt_row0=200) == ESHAPE                                  # d channels past the plane
    assert pvc(ldo=64) == ESHAPE
    assert pvc(Lq=0) == OK
    assert pvc(o=None) == ENULL
    assert pvc(o=A + 2) == EALIGN
    assert pvc(ws=A + 4, wsb=1 << 20) == EALIGN
    # the whole attention: for d = 64 and 128 the workspace holds the codes,
    # flags and scales of Q, K and V^T and their fp8 expansions (256-byte aligned)
    heads, L, d, gs = 2, 256, 128, 16
    al = lambda n: (n + 255) // 256 * 256
    act = lambda rows, k: al(rows * k // 2) + al(rows * k // gs) + al(rows * k // 64 * 2)
    need = 2 * act(heads * L, d) + act(heads * d, L) + 3 * al(heads * L * d)
    assert q.quartz_lzs_attention_workspace_bytes(heads, L, d, gs) == need
    assert q.quartz_lzs_attention_workspace_bytes(heads, 100, d, gs) == 0
    assert q.quartz_lzs_attention_workspace_bytes(heads, L, d, 7) == 0
    la = q.quartz_lzs_attention

    def att(heads=2, L=256, d=128, gs=16, o=A, ldo=256, ws=A, wsb=need):
        return la(A, A, A, heads, L, d, gs, o, ldo, ws, wsb, None)
    assert att(gs=12) == EUNSUP
    assert att(L=100) == ESHAPE
    assert att(L=1 << 17) == ESHAPE                                    # L <= 2^16
    assert att(ldo=128) == ESHAPE                                      # ldo < heads d
    assert att(ldo=258) == EALIGN                                      # ldo % 4
    assert att(heads=0) == OK
    assert att(ws=None) == ENULL
    assert att(o=A + 2) == EALIGN
    assert att(wsb=need - 256) == EWS                                  # nothing launched
