"""GPU parity of the LTP soft-pruning training path (sc_ltp_soft_mask, sc_ltp_soft_backward) against the
CPU oracle, through the C ABI, on seeded inputs.

The GPU forward (window attention, scores) feeds the GPU mask and backward; the oracle recomputes the
whole chain in double precision from the same bf16 inputs and gradients.  Tolerances, from the arithmetic:
  * mask: |gpu - oracle| <= 1e-4 (float32 sigmoid of float32 scores that agree to 1e-5 relative, divided
    by a temperature of the order of the score spread);
  * y (bf16): as the attention output, 2e-2;
  * dq, dk, dv (bf16), per element: |gpu - oracle| <= 4 u scale, u = 2^-8 the unit roundoff of bf16 and scale
    the oracle's error scale of that element (the backward's chain evaluated on magnitudes: every factor by
    its absolute value, every difference by a sum).  A running error bound: every product of the backward
    takes bf16 operands, so each term of a gradient element carries at most two rounded factors (dV: P packed
    and dO = bf16(m dy); dQ, dK: dS packed, whose own inputs dP and D carry the rounding of dO and of the
    forward's stored O, at most u of their magnitude each), the element is stored as bf16 (u of its value,
    itself at most its scale), the mask's relative error reaches the score gradient (below 2^-10 here) and
    float32 accumulation adds n 2^-24 (2^-12 for n = 4096): at most about 3.3 u of the scale in all;
  * dtheta: |gpu - oracle| <= 2u mtheta, mtheta the oracle's scale of dtheta (the sum over tokens of
    (sum |dy out| + |dmask|) m (1 - m) / T): each term carries the rounding of the stored O (u), the mask's
    relative error and float32 accumulation over the tokens.
"""
import numpy as np
import pytest
import torch

import oracle
import sc_inputs as si
from gpu_helpers import check_out, dev_i32, log, make_desc, record, to_dev_storage

pytestmark = pytest.mark.gpu

import paper_2310_07109_amd as sc  # noqa: E402

U_BF16 = 2.0 ** -8
GRAD_K = 4.0
DTH_K = 2.0

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


def check_grad(name, gpu, ref, scale, tag):
    """Per element: |gpu - ref| <= GRAD_K * U_BF16 * scale (the oracle's error scale of the element)."""
    err = np.abs(gpu - ref)
    bound = GRAD_K * U_BF16 * scale
    worst = float((err / np.maximum(bound, 1e-300)).max()) if err.size else 0.0
    nr = float(np.linalg.norm(ref))
    record(f"{tag} {name}: norm rel err {float(np.linalg.norm(gpu - ref)) / max(nr, 1e-30):.3g}, worst err / "
           f"(4u scale) {worst:.3g}")
    assert worst <= 1.0, (name, worst)


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
    rdq, rdk, rdv, rdth, mq, mk, mv, mth = oracle.soft_prune_backward(
        *sel, vl[rows], gp[rows], inp["window"], inp["alpha"], theta, temp, dy64[rows], dm[rows].astype(np.float64),
        kg, scales=True)
    gpu = dict(mask=mask.cpu().numpy()[rows], y=_np(y)[rows], dq=_np(dq)[rows], dk=_np(dk)[rows],
               dv=_np(dv)[rows], dth=float(dth.item()))
    if oracle_rows is not None:  # dtheta sums every sequence: compare the sampled sequences' share instead
        gpu["dth"] = None
    ref = dict(mask=rm, y=ry, dq=rdq, dk=rdk, dv=rdv, dth=rdth, mq=mq, mk=mk, mv=mv, mth=mth)
    return gpu, ref


def compare(gpu, ref, valid_len, tag):
    assert np.all(np.abs(gpu["mask"] - ref["mask"]) <= 1e-4), float(np.abs(gpu["mask"] - ref["mask"]).max())
    check_out(gpu["y"], ref["y"], "bf16", what="y")
    for key, mkey in (("dq", "mq"), ("dk", "mk"), ("dv", "mv")):
        check_grad(key, gpu[key], ref[key], ref[mkey], tag)
        for b in range(len(valid_len)):
            assert np.all(gpu[key][b, valid_len[b]:] == 0.0), key
    if gpu["dth"] is not None:
        e = abs(gpu["dth"] - ref["dth"])
        record(f"{tag} dtheta: gpu {gpu['dth']:.7g} oracle {ref['dth']:.7g}, rel err "
               f"{e / max(abs(ref['dth']), 1e-30):.3g}, err / (2u scale) {e / max(DTH_K * U_BF16 * ref['mth'], 1e-300):.3g}")
        assert e <= DTH_K * U_BF16 * ref["mth"] + 1e-9


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
    compare(gpu, ref, inp["valid_len"], f"soft {name}")


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
    compare(gpu, ref, inp["valid_len"], "soft globals on the slope")


def test_soft_config4_all_sequences():
    """The B8 n4096 H12 window-512 32-global workload on the GPU (the launch configuration of the benchmark),
    every sequence through the oracle, dtheta over the whole batch."""
    inp = si.make_attention_inputs(si.CONFIGS[4])
    gpu, ref = run_soft(inp, 1)
    compare(gpu, ref, inp["valid_len"], "soft config 4")


def test_soft_backward_deterministic():
    cfg = si.AttnConfig("det", 18, 2, 400, 2, 64, "bf16", 64, (300, 400), 4, "random", input_scale=1.0)
    inp = si.make_attention_inputs(cfg)
    a, _ = run_soft(inp, 1)
    b, _ = run_soft(inp, 1)
    for key in ("mask", "y", "dq", "dk", "dv"):
        assert np.array_equal(a[key], b[key]), key
    assert a["dth"] == b["dth"]
