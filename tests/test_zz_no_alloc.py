"""sc_window_attention_noalloc (the window attention with the library's static device workspace, for callers
that cannot allocate) against sc_window_attention (caller's workspace), through the C ABI: the same kernels on
the same inputs, so every output must be bit-identical.  Two calls in a row, the second on a smaller problem
(the static workspace keeps the first call's contents)."""
import numpy as np
import pytest
import torch

import sc_inputs as si
from gpu_helpers import log, make_desc, to_dev_storage

import paper_2310_07109_amd as sc

pytestmark = pytest.mark.gpu


def _outputs(inp, noalloc, band=False):
    d = make_desc(inp)
    q, k, v = (to_dev_storage(inp[x], inp["dtype"]) for x in ("q", "k", "v"))
    out = torch.full_like(q, float("nan"))
    lse = torch.full((d.B, d.H, d.n), float("nan"), dtype=torch.float32, device=q.device)
    sp = torch.full((sc.sc_score_partials_size(d) // 4,), float("nan"), dtype=torch.float32, device=q.device)
    bp = torch.full((sc.sc_band_probs_size(d) // 4,), float("nan"), dtype=torch.float32, device=q.device) \
        if band else None
    if noalloc:
        sc.sc_window_attention_noalloc(d, q, k, v, out, lse, sp, bp)
    else:
        sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, band_probs=bp if band else False)
    scores = sc.sc_ltp_score(d, sp)
    torch.cuda.synchronize()
    res = dict(out=out.view(torch.int16 if inp["dtype"] == "bf16" else torch.int32).cpu().numpy(),
               lse=lse.cpu().numpy(), scores=scores.cpu().numpy())
    if band:
        res["band"] = bp.cpu().numpy()
    return res


def _same(a, b, what):
    for key in a:
        assert np.array_equal(a[key], b[key], equal_nan=True), f"{what}: {key} differs"


def test_noalloc_matches_workspace_entry_point_twice():
    big = si.make_attention_inputs(si.CONFIGS[4], B=4, n=4096)
    small = si.make_attention_inputs(si.CONFIGS[4], seed=13, B=2, n=700, H=4, window=128, n_global=3,
                                     len_range=(500, 700))
    log(f"no-alloc: workspace {sc.sc_window_attention_workspace_size(make_desc(big))} bytes, then "
        f"{sc.sc_window_attention_workspace_size(make_desc(small))} bytes, of {sc.SC_NOALLOC_SCRATCH_BYTES}")
    for name, inp in (("B4 n4096 w512 G32", big), ("B2 n700 w128 G3", small)):
        ref = _outputs(inp, noalloc=False)
        got = _outputs(inp, noalloc=True)
        _same(ref, got, name)
        log(f"no-alloc {name}: bit-identical")
    # the paper's band layout through the static workspace as well (small problem)
    _same(_outputs(small, noalloc=False, band=True), _outputs(small, noalloc=True, band=True), "band layout")


def test_noalloc_rejects_oversized_problem():
    """A problem whose workspace exceeds the static buffer is refused on the host; nothing is enqueued (the
    tensor pointers are never used)."""
    import ctypes
    B, n, G = 64, 4096, 64
    vl = torch.full((B,), n, dtype=torch.int32, device="cuda:0")
    gp = torch.zeros((B, G), dtype=torch.int32, device="cuda:0")
    d = sc.Desc(B, n, 16, 512, vl, gp, 0.125, sc.SC_BF16)
    assert sc.sc_window_attention_workspace_size(d) > sc.SC_NOALLOC_SCRATCH_BYTES
    p = vl.data_ptr()
    rc = sc.load().sc_window_attention_noalloc(ctypes.byref(d.c()), p, p, p, p, None, None, None,
                                               ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == sc.SC_ENOSCRATCH
