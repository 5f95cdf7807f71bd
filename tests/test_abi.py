"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/sc.h, sizes its buffers consistently, and rejects invalid
arguments on the host before touching the device."""
import ctypes
import os
import re

import pytest

import paper_2310_07109_amd as sc
from paper_2310_07109_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sc.h")

pytestmark = pytest.mark.skipif(not os.path.exists(sc.lib_path()), reason="libsc.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sc_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = sc.load()
    names = declared_functions()
    assert len(names) == 21
    for name in names:
        assert hasattr(L, name), name


@pytest.mark.skipif(not os.path.exists(sc.debug_lib_path()), reason="libsc_debug.so not built")
def test_debug_library_exports_the_same_entry_points():
    L = sc.load_debug()
    for name in declared_functions():
        assert hasattr(L, name), name
    # its host-side checks are the release library's (nothing reaches the device-side check or a launch)
    assert L.sc_window_attention(ctypes.byref(desc(d=32).c()), 0x100000, 0x200000, 0x300000, 0x400000, None, None,
                                 None, None, 0, None) == B.SC_EUNSUPPORTED
    assert L.sc_window_attention(ctypes.byref(desc().c()), None, 0x200000, 0x300000, 0x400000, None, None, None,
                                 None, 0, None) in (B.SC_EINVAL, B.SC_EHIP)


def test_validate_desc_host_checks():
    """sc_validate_desc rejects on the host (no launch) a null result word and an invalid descriptor."""
    L = sc.load()
    assert L.sc_validate_desc(ctypes.byref(desc().c()), None, None) == B.SC_EINVAL
    assert L.sc_validate_desc(ctypes.byref(desc(B=0).c()), 0x700000, None) == B.SC_EINVAL
    assert L.sc_validate_desc(ctypes.byref(desc(G=3).c()), 0x700000, None) == B.SC_EINVAL
    assert L.sc_validate_desc(ctypes.byref(desc(d=32).c()), 0x700000, None) == B.SC_EUNSUPPORTED
    assert L.sc_validate_desc(None, 0x700000, None) == B.SC_EINVAL


def test_status_strings():
    assert sc.sc_status_str(0) == "ok"
    for code in (-1, -2, -3, -4, -5):
        assert sc.sc_status_str(code) not in ("ok", "unknown status")


class FakeT:
    """Stands in for a device tensor: only an address (never dereferenced)."""

    def __init__(self, addr):
        self.addr = addr

    def data_ptr(self):
        return self.addr


def desc(**kw):
    base = dict(B=2, n=256, H=4, window=64, valid_len=FakeT(0x10000), global_pos=None, softmax_scale=0.125,
                dtype=B.SC_BF16)
    base.update(kw)
    gp = base.pop("global_pos")
    G = base.pop("G", 0)
    d = sc.Desc(**base)
    d.global_pos, d.G = gp, G
    return d


def call_attn(d, q=0x100000, k=0x200000, v=0x300000, out=0x400000, lse=None, ws=None, ws_bytes=0):
    L = sc.load()
    return L.sc_window_attention(ctypes.byref(d.c()), q, k, v, out, lse, None, None, ws, ws_bytes, None)


def test_invalid_descriptors_rejected_before_launch():
    assert call_attn(desc(d=32)) == B.SC_EUNSUPPORTED
    assert call_attn(desc(window=-1)) == B.SC_EINVAL
    assert call_attn(desc(B=0)) == B.SC_EINVAL
    assert call_attn(desc(n=0)) == B.SC_EINVAL
    assert call_attn(desc(H=0)) == B.SC_EINVAL
    assert call_attn(desc(dtype=7)) == B.SC_EINVAL
    assert call_attn(desc(softmax_scale=float("nan"))) == B.SC_EINVAL
    assert call_attn(desc(softmax_scale=float("inf"))) == B.SC_EINVAL
    assert call_attn(desc(softmax_scale=-0.125)) == B.SC_EINVAL
    assert call_attn(desc(valid_len=None)) == B.SC_EINVAL
    # G > 0 needs global positions, and G may not exceed n
    assert call_attn(desc(G=3)) == B.SC_EINVAL
    assert call_attn(desc(global_pos=FakeT(0x50000), G=257)) == B.SC_EINVAL


def test_causal_flag_checked():
    assert call_attn(desc(causal=True, dtype=B.SC_F32)) == B.SC_EUNSUPPORTED
    L = sc.load()
    bad = desc()
    c = bad.c()
    c.causal = 2
    assert L.sc_window_attention(ctypes.byref(c), 0x100000, 0x200000, 0x300000, 0x400000, None, None, None,
                                 0x900000, 1 << 30, None) == B.SC_EINVAL
    c = desc(causal=True).c()
    assert L.sc_window_attention(ctypes.byref(c), 0x100000, 0x200000, 0x300000, 0x400000, None, None, 0x800000,
                                 0x900000, 1 << 30, None) == B.SC_EUNSUPPORTED   # band layout not with causal


def test_null_and_aliasing_rejected():
    d = desc()
    assert call_attn(d, q=None) == B.SC_EINVAL
    assert call_attn(d, out=None) == B.SC_EINVAL
    # out overlapping q (tensor is 2*256*4*64*2 bytes = 256 KiB)
    assert call_attn(d, out=0x100000 + 4096) == B.SC_EINVAL
    assert call_attn(d, lse=0x400000 + 64) == B.SC_EINVAL


def test_workspace_checked():
    d = desc(global_pos=FakeT(0x50000), G=4)
    need = sc.sc_window_attention_workspace_size(d)
    assert need > 0
    assert call_attn(d, ws=None, ws_bytes=0) == B.SC_EWORKSPACE
    assert call_attn(d, ws=0x900000, ws_bytes=need - 1) == B.SC_EWORKSPACE
    # without global tokens only the per-row log2-LSE handed from pass 1 to pass 2 remains
    assert sc.sc_window_attention_workspace_size(desc()) == 4 * 2 * 4 * 256


def test_sizes():
    d = desc()
    # partials: per (b, h): n band column sums + ceil(n/512) * G global columns + ceil(G/64) * n global-row sums
    assert sc.sc_score_partials_size(d) == 4 * 2 * 4 * 256
    dg = desc(global_pos=FakeT(0x50000), G=3)
    assert sc.sc_score_partials_size(dg) == 4 * 2 * 4 * (256 + 1 * 3 + 1 * 256)
    # band layout: [B,H,n,2r+1] + [B,H,n,G] + [B,H,G,n]
    assert sc.sc_band_probs_size(dg) == 4 * 2 * 4 * 256 * (65 + 2 * 3)
    # huge window: r clamps to n - 1 for the band layout
    assert sc.sc_band_probs_size(desc(window=10 ** 6)) == 4 * 2 * 4 * 256 * (2 * 255 + 1)
    assert sc.sc_score_partials_size(desc(d=16)) == 0
    # band-mode score workspace: the partials plus, per (b, h) and block of 128 rows, the 128 + 2r keys the block
    # reaches, rounded up to 256
    assert sc.sc_ltp_score_workspace_size(dg, sc.SC_SCORE_FROM_PARTIALS) == 0
    assert sc.sc_ltp_score_workspace_size(dg, sc.SC_SCORE_FROM_BAND_PROBS) == \
        sc.sc_score_partials_size(dg) + 4 * 2 * 4 * 2 * 256
    wide = desc(window=10 ** 6)
    assert sc.sc_ltp_score_workspace_size(wide, sc.SC_SCORE_FROM_BAND_PROBS) == \
        sc.sc_score_partials_size(wide) + 4 * 2 * 4 * 2 * 768
    assert sc.sc_encoder_attn_stack_workspace_size(desc(), 3) > 0
    assert sc.sc_encoder_attn_stack_workspace_size(desc(), 0) == 0


def test_prune_validation():
    L = sc.load()
    d = desc()
    cd = d.c()
    ws_need = sc.sc_ltp_prune_compact_workspace_size(d)
    assert ws_need == 4 * 2 * 256

    def call(scores=0x100000, nt=0, src=None, dst=None, rb=None, keep=0x200000, nl=0x300000, ws=0x800000,
             wsb=ws_need, oin=None, oout=None):
        return L.sc_ltp_prune_compact(ctypes.byref(cd), scores, ctypes.c_float(0.01), 1, nt, src, dst, rb, keep, nl,
                                      None, oin, oout, ws, wsb, None)

    assert call(scores=None) == B.SC_EINVAL
    assert call(keep=None) == B.SC_EINVAL
    assert call(nt=5) == B.SC_EINVAL
    assert call(nt=1) == B.SC_EINVAL  # arrays missing
    assert call(ws=None) == B.SC_EWORKSPACE
    assert call(wsb=ws_need - 4) == B.SC_EWORKSPACE
    one = lambda x: (ctypes.c_void_p * 1)(x)  # noqa: E731
    rb = (ctypes.c_int64 * 1)(128)
    assert call(nt=1, src=one(0x1000000), dst=one(0x1000000 + 128), rb=rb) == B.SC_EINVAL  # src/dst overlap
    assert call(nt=1, src=one(0x1000000), dst=one(0x2000000), rb=(ctypes.c_int64 * 1)(0)) == B.SC_EINVAL
    assert call(oin=0x3000000, oout=0x3000000 + 8) == B.SC_EINVAL


def test_topk_validation():
    L = sc.load()
    cd = desc().c()
    ws_need = sc.sc_ltp_prune_compact_workspace_size(desc())

    def call(ratio, ws=0x800000):
        return L.sc_topk_prune_compact(ctypes.byref(cd), 0x100000, ctypes.c_float(ratio), 1, 0, None, None, None,
                                       0x200000, 0x300000, None, None, None, ws, ws_need, None)

    for bad in (-0.01, 1.01, float("nan"), float("inf")):
        assert call(bad) == B.SC_EINVAL
    assert call(0.5, ws=None) == B.SC_EWORKSPACE


def test_soft_pruning_validation():
    """Every call here is rejected on the host (nothing is launched on the fake addresses)."""
    L = sc.load()
    d = desc()
    cd = d.c()
    A = [0x1000000 * (i + 1) for i in range(12)]  # disjoint fake device buffers

    def fwd(scores=A[0], theta=0.01, t=0.01, out=A[1], mask=A[2], y=A[3], dd=cd):
        return L.sc_ltp_soft_mask(ctypes.byref(dd), scores, ctypes.c_float(theta), ctypes.c_float(t), 1, out, mask,
                                  y, None)

    assert fwd(scores=None) == B.SC_EINVAL
    assert fwd(t=0.0) == B.SC_EINVAL
    assert fwd(t=-1.0) == B.SC_EINVAL
    assert fwd(theta=float("nan")) == B.SC_EINVAL
    assert fwd(y=A[1] + 64) == B.SC_EINVAL  # y overlaps out
    f32 = desc(dtype=B.SC_F32)
    assert fwd(dd=f32.c()) == B.SC_EUNSUPPORTED
    causal = desc(causal=True)
    assert fwd(dd=causal.c()) == B.SC_EUNSUPPORTED
    ws_need = sc.sc_ltp_soft_backward_workspace_size(d)
    assert ws_need > 0 and sc.sc_ltp_soft_backward_workspace_size(f32) == 0

    def bwd(dq=A[7], dk=A[8], dv=A[9], dth=A[10], ws=A[11], wsb=ws_need, t=0.01, q=A[0]):
        return L.sc_ltp_soft_backward(ctypes.byref(cd), q, A[1], A[2], A[3], A[4], A[5], ctypes.c_float(t), 1,
                                      A[6], None, dq, dk, dv, dth, ws, wsb, None)

    assert bwd(q=None) == B.SC_EINVAL
    assert bwd(dth=None) == B.SC_EINVAL
    assert bwd(t=0.0) == B.SC_EINVAL
    assert bwd(ws=None) == B.SC_EWORKSPACE
    assert bwd(wsb=ws_need - 1) == B.SC_EWORKSPACE
    assert bwd(dq=A[0] + 128) == B.SC_EINVAL  # dq overlaps q
    assert bwd(dk=A[7] + 128) == B.SC_EINVAL  # dk overlaps dq
    assert bwd(dth=A[11] + 4) == B.SC_EINVAL  # dtheta inside the workspace


def test_full_stack_validation():
    L = sc.load()
    cd = desc().c()
    w = (ctypes.c_void_p * 1)(0x5000000)
    th = (ctypes.c_float * 1)(0.0)

    def call(W1=w, W2=w, F=64, windows=None, ws=0x900000):
        return L.sc_encoder_stack(ctypes.byref(cd), 1, windows, 0x100000, w, w, W1, W2, F, th, 1,
                                  ctypes.c_float(1e-5), 0x200000, 0x300000, None, None, ws, 1 << 30, None)

    assert call(W1=None) == B.SC_EINVAL
    assert call(W2=None) == B.SC_EINVAL
    assert call(F=0) == B.SC_EINVAL
    assert call(F=12) == B.SC_EINVAL                       # not a multiple of 8
    assert call(windows=(ctypes.c_int32 * 1)(-1)) == B.SC_EINVAL
    assert call(ws=None) == B.SC_EWORKSPACE
    d = desc()
    assert sc.sc_encoder_stack_workspace_size(d, 2, 3072) > sc.sc_encoder_attn_stack_workspace_size(d, 2)
    assert sc.sc_encoder_stack_workspace_size(d, 2, 0) == 0


def test_score_and_stack_validation():
    L = sc.load()
    d = desc()
    cd = d.c()
    assert L.sc_ltp_score(ctypes.byref(cd), 5, 0x100000, 0x200000, None, 0, None) == B.SC_EINVAL
    assert L.sc_ltp_score(ctypes.byref(cd), 0, None, 0x200000, None, 0, None) == B.SC_EINVAL
    dd = desc(dtype=B.SC_F32)
    w = (ctypes.c_void_p * 1)(0x5000000)
    th = (ctypes.c_float * 1)(0.0)
    assert L.sc_encoder_attn_stack(ctypes.byref(dd.c()), 1, 0x100000, w, w, th, 1, ctypes.c_float(1e-5), 0x200000,
                                   0x300000, None, None, 0x900000, 1 << 30, None) == B.SC_EUNSUPPORTED
    assert L.sc_encoder_attn_stack(ctypes.byref(cd), 1, 0x100000, w, w, th, 1, ctypes.c_float(0.0), 0x200000,
                                   0x300000, None, None, 0x900000, 1 << 30, None) == B.SC_EINVAL
    assert L.sc_encoder_attn_stack(ctypes.byref(cd), 1, 0x100000, w, w, th, 1, ctypes.c_float(1e-5), 0x200000,
                                   0x300000, None, None, None, 0, None) == B.SC_EWORKSPACE
    # the products pack the surviving rows of all sequences with a per-workgroup prefix table: B <= 8192
    wide = desc(B=8193, n=16, H=2, window=4, G=0)
    assert L.sc_encoder_attn_stack(ctypes.byref(wide.c()), 1, 0x100000, w, w, th, 1, ctypes.c_float(1e-5),
                                   0x200000, 0x300000, None, None, 0x900000, 1 << 30, None) == B.SC_EUNSUPPORTED


def test_noalloc_rejects_oversized_problems_on_the_host():
    """The no-allocation window attention refuses a problem whose workspace exceeds its static buffer, and an
    invalid descriptor, before any device call."""
    L = sc.load()
    big = desc(B=64, n=4096, H=16, window=512, G=64, global_pos=FakeT(0x20000))
    assert L.sc_window_attention_workspace_size(ctypes.byref(big.c())) > B.SC_NOALLOC_SCRATCH_BYTES
    rc = L.sc_window_attention_noalloc(ctypes.byref(big.c()), 0x100000, 0x200000, 0x300000, 0x400000, None, None,
                                       None, None)
    assert rc == B.SC_ENOSCRATCH
    bad = desc(d=32)
    rc = L.sc_window_attention_noalloc(ctypes.byref(bad.c()), 0x100000, 0x200000, 0x300000, 0x400000, None, None,
                                       None, None)
    assert rc == B.SC_EUNSUPPORTED
