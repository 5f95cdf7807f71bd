"""GPU parity of the LTP soft-pruning training path (sc_ltp_soft_mask, sc_ltp_soft_backward) against the
CPU oracle, through the C ABI, on seeded inputs.

The GPU forward (window attention, scores) feeds the GPU mask and backward; the oracle recomputes the
whole chain in double precision from the same bf16 inputs and gradients.  Tolerances, from the arithmetic:
  * mask: |gpu - oracle| <= 1e-4 (float32 sigmoid of float32 scores that agree to 1e-5 relative, divided
    by a temperature of the order of the score spread);
  * y (bf16): as the attention output, 2e-2;
  * dq, dk, dv (bf16): every product runs on bf16 operands (dO = bf16(m dy), P and dS rounded to bf16 for
    the MFMAs, the forward's O stored as bf16), each a relative perturbation of 2^-9 of its terms, and the
    result is stored as bf16 (2^-9); a handful of such roundings, with the cancellation of dP - D in dS
    amplifying them a few times, stays within 2^-6 in the norm of each tensor and 2^-5 of its largest
    element per element;
  * dtheta: a float32 sum of the score gradients of every token, each perturbed by the bf16 output it
    is taken against; the terms have both signs, so the bound is 2^-6 of the sum of their magnitudes.
"""
import numpy as np
import pytest
import torch

import oracle
import sc_inputs as si
from gpu_helpers import check_out, dev_i32, log, make_desc, to_dev_storage

pytestmark = pytest.mark.gpu

import paper_2310_07109_amd as sc  # noqa: E402

NORM_TOL = 2.0 ** -6
ELEM_TOL = 2.0 ** -5

CASES = [
    # name, B, n, H, window, G, lengths (None: uniform over range), range, input scale, keep_global
    ("ragged with globals", 2, 300, 2, 64, 3, None, (200, 300), 1.0, 1),
    ("globals pruned softly", 2, 300, 2, 64, 3, None, (200, 300), 1.0, 0),
    ("two global chunks, two spans", 1, 700, 2, 128, 70, None, (650, 700), 0.5, 1),
    ("empty and single-token sequences", 3, 200, 2, 16, 2, [0, 1, 200], (0, 200), 1.0, 1),
    ("no globals, window wider than the sequence", 2, 513, 3, 1000, 0, None, (400, 513), 0.5, 1),
    ("three spans", 1, 1300, 2, 256, 5, None, (1200, 1300), 1.0, 1),
    ("all tokens global", 1, 96, 2, 8, 96, None, (96, 96), 1.0, 1),
    ("window 0", 2, 100, 2, 0, 1, None, (60, 100), 1.0, 1),
]


def _bf16_t(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda:0").view(torch.bfloat16)


def _np(t):
    return t.float().cpu().numpy().astype(np.float64)


def check_grad(name, gpu, ref):
    nr = float(np.linalg.norm(ref))
    err = float(np.linalg.norm(gpu - ref))
    emax = float(np.abs(gpu - ref).max()) if ref.size else 0.0
    amax = float(np.abs(ref).max()) if ref.size else 0.0
    log(f"  {name}: norm rel err {err / max(nr, 1e-30):.3g}, max err / max {emax / max(amax, 1e-30):.3g}")
    assert err <= NORM_TOL * nr + 1e-30, (name, err, nr)
    assert emax <= ELEM_TOL * amax + 1e-30, (name, emax, amax)


def run_soft(inp, kg, seed=21, theta_at_globals=False, oracle_rows=None):
    """GPU forward + backward and the oracle's; returns both sides' results.  theta_at_globals: the threshold
    and temperature are taken from the global tokens' scores (so their soft masks are on the sigmoid's slope
    when keep_global is 0).  oracle_rows: run the oracle on these sequences only (they are independent)."""
    B, n, H, d = inp["B"], inp["n"], inp["H"], inp["d"]
    dsc = make_desc(inp)
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    out, lse, sp, _ = sc.sc_window_attention(dsc, q, k, v, lse=True, score_partials=True)
    scores = sc.sc_ltp_score(dsc, sp)
    s_np = scores.cpu().numpy().astype(np.float64)
    vl, gp = inp["valid_len"], inp["global_pos"]
    vals = []
    for b in range(B):
        g = {int(p) for p in gp[b] if 0 <= p < vl[b]}
        vals.extend(s_np[b, t] for t in range(vl[b]) if (t in g) == theta_at_globals)
    theta = float(np.median(vals)) if vals else 0.0
    temp = max(float(np.std(vals)) if vals else 0.0, 1e-6)
    mask, y = sc.sc_ltp_soft_mask(dsc, scores, theta, temp, out, keep_global=bool(kg))
    dy_s, dy64, dm = si.make_soft_gradients(seed, B, n, H, d)
    dy = _bf16_t(dy_s)
    dmask = torch.from_numpy(dm).to("cuda:0")
    dq, dk, dv, dth = sc.sc_ltp_soft_backward(dsc, q, k, v, out, lse, mask, temp, dy, dmask, keep_global=bool(kg))
    torch.cuda.synchronize()
    rows = np.arange(B) if oracle_rows is None else np.asarray(oracle_rows)
    sel = [inp[x][rows] for x in ("q64", "k64", "v64")]
    ro, rl, rs, rm, ry = oracle.soft_prune_forward(*sel, vl[rows], gp[rows], inp["window"], inp["alpha"], theta,
                                                   temp, kg)
    rdq, rdk, rdv, rdth = oracle.soft_prune_backward(*sel, vl[rows], gp[rows], inp["window"], inp["alpha"], theta,
                                                     temp, dy64[rows], dm[rows].astype(np.float64), kg)
    gpu = dict(mask=mask.cpu().numpy()[rows], y=_np(y)[rows], dq=_np(dq)[rows], dk=_np(dk)[rows],
               dv=_np(dv)[rows], dth=float(dth.item()))
    if oracle_rows is not None:  # dtheta sums every sequence: compare the sampled sequences' share instead
        gpu["dth"] = None
    # scale of dtheta's error: the sum of the magnitudes of the terms it adds (it cancels)
    dmk = (dy64[rows] * ro).sum(axis=(2, 3)) + dm[rows].astype(np.float64)
    terms = np.abs(dmk * rm * (1.0 - rm)) / temp
    for i, b in enumerate(rows):
        terms[i, vl[b]:] = 0.0
        if kg:
            for p in gp[b]:
                if 0 <= p < vl[b]:
                    terms[i, p] = 0.0
    ref = dict(mask=rm, y=ry, dq=rdq, dk=rdk, dv=rdv, dth=rdth, dth_abs=float(terms.sum()))
    return gpu, ref


def compare(gpu, ref, valid_len):
    assert np.all(np.abs(gpu["mask"] - ref["mask"]) <= 1e-4), float(np.abs(gpu["mask"] - ref["mask"]).max())
    check_out(gpu["y"], ref["y"], "bf16", what="y")
    for key in ("dq", "dk", "dv"):
        check_grad(key, gpu[key], ref[key])
        for b in range(len(valid_len)):
            assert np.all(gpu[key][b, valid_len[b]:] == 0.0), key
    if gpu["dth"] is not None:
        log(f"  dtheta gpu {gpu['dth']:.6g} oracle {ref['dth']:.6g} (sum of |terms| {ref['dth_abs']:.6g})")
        assert abs(gpu["dth"] - ref["dth"]) <= NORM_TOL * ref["dth_abs"] + 1e-6


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_soft_small_cases(case):
    name, B, n, H, window, G, lens, lr, scale, kg = case
    log(f"soft case {name}")
    cfg = si.AttnConfig(name, 17, B, n, H, 64, "bf16", window, lr, G, "random", input_scale=scale)
    inp = si.make_attention_inputs(cfg)
    if lens is not None:
        inp["valid_len"] = np.array(lens, np.int32)
        inp["global_pos"] = si.global_positions(17, inp["valid_len"], G, "random")
    gpu, ref = run_soft(inp, kg)
    compare(gpu, ref, inp["valid_len"])


def test_soft_global_tokens_on_the_slope():
    """keep_global 0 with the threshold among the global tokens' scores: their masks and score gradients count."""
    cfg = si.AttnConfig("globals on the slope", 19, 2, 400, 2, 64, "bf16", 32, (300, 400), 6, "random",
                        input_scale=1.0)
    inp = si.make_attention_inputs(cfg)
    gpu, ref = run_soft(inp, 0, theta_at_globals=True)
    m = ref["mask"]
    on_slope = sum(1 for b in range(inp["B"]) for p in inp["global_pos"][b]
                   if 0 <= p < inp["valid_len"][b] and 0.05 < m[b, p] < 0.95)
    log(f"  global tokens with 0.05 < mask < 0.95: {on_slope}")
    assert on_slope >= 3
    compare(gpu, ref, inp["valid_len"])


def test_soft_config4_sampled_sequences():
    """The B8 n4096 H12 window-512 32-global workload on the GPU (the launch configuration of the benchmark);
    three of its sequences (among them the longest) through the oracle."""
    inp = si.make_attention_inputs(si.CONFIGS[4])
    rows = [0, 2, 5]
    gpu, ref = run_soft(inp, 1, oracle_rows=rows)
    compare(gpu, ref, inp["valid_len"][rows])


def test_soft_backward_deterministic():
    cfg = si.AttnConfig("det", 18, 2, 400, 2, 64, "bf16", 64, (300, 400), 4, "random", input_scale=1.0)
    inp = si.make_attention_inputs(cfg)
    a, _ = run_soft(inp, 1)
    b, _ = run_soft(inp, 1)
    for key in ("mask", "y", "dq", "dk", "dv"):
        assert np.array_equal(a[key], b[key]), key
    assert a["dth"] == b["dth"]
