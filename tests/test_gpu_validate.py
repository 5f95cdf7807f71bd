"""sc_validate_desc, the device-side check of a descriptor's valid_len and global_pos (which the host cannot
read and the kernels clamp or ignore when out of range), and libsc_debug.so, the library built with SC_DEBUG,
which runs that check before every call: invalid device inputs are refused with SC_EINVAL before anything else
is enqueued, and valid ones give the release library's results bit for bit.  All through the C ABI."""
import ctypes

import numpy as np
import pytest
import torch

import sc_inputs as si
from gpu_helpers import dev_i32, log, make_desc, to_dev_storage

import paper_2310_07109_amd as sc
from paper_2310_07109_amd import _binding as B

pytestmark = pytest.mark.gpu

V_LEN, V_RANGE, V_ORDER, V_FIRST = sc.SC_VALID_LEN, sc.SC_VALID_POS_RANGE, sc.SC_VALID_POS_ORDER, \
    sc.SC_VALID_POS_UNUSED_FIRST

# (lengths, global positions or None, expected bits); B = 2 sequences, n = 16
CASES = [
    ([16, 5], [[0, 3, 9], [1, 4, -1]], 0),
    ([16, 0], [[0, 3, 9], [-1, -1, -1]], 0),
    ([16, 5], None, 0),
    ([-1, 5], [[0, 3, 9], [1, 4, -1]], V_LEN | V_RANGE),  # positions are also checked against the raw length
    ([-1, 5], None, V_LEN),
    ([17, 5], None, V_LEN),
    ([16, 5], [[0, 3, 9], [1, 5, -1]], V_RANGE),      # a position at its sequence's length
    ([16, 5], [[0, -2, -1], [1, 4, -1]], V_RANGE),    # below -1
    ([16, 5], [[3, 0, 9], [1, 4, -1]], V_ORDER),      # descending
    ([16, 5], [[3, 3, 9], [1, 4, -1]], V_ORDER),      # repeated
    ([16, 5], [[-1, 3, 9], [1, 4, -1]], V_FIRST),     # a used slot after an unused one
    ([20, 5], [[0, 3, 9], [2, 1, -1]], V_LEN | V_ORDER),
    ([16, 3], [[0, 3, 9], [4, 1, 7]], V_RANGE | V_ORDER),
]


@pytest.mark.parametrize("lens,gpos,want", CASES)
def test_validate_desc_bits(lens, gpos, want):
    vl = dev_i32(np.array(lens, dtype=np.int32))
    gp = dev_i32(np.array(gpos, dtype=np.int32)) if gpos is not None else None
    d = sc.Desc(2, 16, 2, 8, vl, gp)
    got = int(sc.sc_validate_desc(d).item())
    assert got == want, (lens, gpos, got, want)


def test_validate_desc_on_the_workloads():
    for cid in (2, 4, 6):
        inp = si.make_attention_inputs(si.CONFIGS[cid])
        assert int(sc.sc_validate_desc(make_desc(inp)).item()) == 0, cid


def _attention(lib, d, q, k, v):
    """One window-attention call through `lib` (the release or the debug library); returns its status and the
    outputs (O as raw bits, LSE, score partials), all initialised to NaN."""
    out = torch.full_like(q, float("nan"))
    lse = torch.full((d.B, d.H, d.n), float("nan"), dtype=torch.float32, device=q.device)
    sp = torch.full((sc.sc_score_partials_size(d) // 4,), float("nan"), dtype=torch.float32, device=q.device)
    wsb = sc.sc_window_attention_workspace_size(d)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    cd = d.c()
    vp = ctypes.c_void_p
    st = lib.sc_window_attention(ctypes.byref(cd), vp(q.data_ptr()), vp(k.data_ptr()), vp(v.data_ptr()),
                                 vp(out.data_ptr()), vp(lse.data_ptr()), vp(sp.data_ptr()), None, vp(ws.data_ptr()),
                                 ctypes.c_size_t(wsb), vp(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    return st, out.view(torch.int16).cpu().numpy(), lse.cpu().numpy(), sp.cpu().numpy()


def test_debug_library_matches_release_and_refuses_invalid_lengths():
    rel, dbg = sc.load(), sc.load_debug()
    inp = si.make_attention_inputs(si.CONFIGS[2], B=3, n=640, len_range=(300, 640))
    d = make_desc(inp)
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    st_r, o_r, l_r, p_r = _attention(rel, d, q, k, v)
    st_d, o_d, l_d, p_d = _attention(dbg, d, q, k, v)
    assert st_r == 0 and st_d == 0
    assert np.array_equal(o_r, o_d) and np.array_equal(l_r, l_d, equal_nan=True)
    assert np.array_equal(p_r, p_d, equal_nan=True)
    # a length beyond n: the debug build refuses the call before enqueueing the attention
    bad = np.array(inp["valid_len"], dtype=np.int32)
    bad[1] = d.n + 1
    dbad = sc.Desc(d.B, d.n, d.H, d.window, dev_i32(bad), d.global_pos, d.softmax_scale, d.dtype)
    st_b, o_b, l_b, p_b = _attention(dbg, dbad, q, k, v)
    assert st_b == B.SC_EINVAL
    nan_bits = torch.full_like(q, float("nan")).view(torch.int16).cpu().numpy()
    assert np.array_equal(o_b, nan_bits) and np.isnan(l_b).all() and np.isnan(p_b).all(), \
        "nothing may be written when the call is refused"
    log(f"debug build: bit-identical outputs on {d.B} sequences, invalid length refused (status {st_b})")
