"""Shared pieces of the GPU parity tests: moving seeded inputs to the device,
running the HIP path through the C ABI, and the comparison rules.

Tolerances (fixed by the workload specification):
  * float32 outputs (O, LSE): |gpu - oracle| <= 1e-4 * |oracle| + 1e-6 * rms(oracle)
  * bfloat16 outputs (O, hidden states): |gpu - oracle| <= 2e-2
  * hidden states of the stacks (stored as bf16 after LayerNorm): 2e-2 plus one bf16 step at the oracle's
    value (the spacing 2^(floor(log2 |v|) - 7)).  The two sides accumulate in different orders, so a value
    near a rounding midpoint can be stored one bf16 step away, and a bf16 step exceeds 2e-2 for values beyond
    4 (LayerNorm outputs reach them).  Full layers add two more bf16 storage points (the attention sub-layer output and the GELU
    activations).  The number of elements beyond 2e-2 is returned for the run's record
  * LSE is computed in float32 in both modes and follows the float32 rule
  * scores (float32 reductions of float32 probabilities from the same inputs):
    |gpu - oracle| <= 1e-5 * |oracle|, exactly 0 beyond the valid length
  * kept-token lists: bit-exact, except tokens whose oracle score lies within
    1e-6 of the threshold, which are excluded and counted.  When both sides score
    the same inputs (single-layer calls), a disagreement is further allowed only
    where the GPU score, within the score tolerance of the oracle's, can lie on the
    other side of the threshold: |s_oracle - theta| <= 1e-5 |s_oracle|.  Counts of
    exclusions and disagreements are asserted and recorded for the run's summary.
"""
import json
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2310_07109_amd as sc  # noqa: E402

DEV = "cuda:0"
NEAR_THETA = 1e-6
SCORE_REL = 1e-5


def log(msg):
    print(msg, flush=True)


def record(msg):
    """A line for the terminal summary of the run (shown even with -q)."""
    from conftest import RECORDS
    RECORDS.append(msg)
    log(msg)


def stored_threshold(cfg_id):
    with open(os.path.join(ROOT, "tests", "golden", "thresholds.json")) as f:
        return json.load(f)[str(cfg_id)]["theta"]


def to_dev_storage(arr, dtype):
    """numpy storage array (uint16 bf16 bits or float32) -> device tensor of the storage dtype."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(DEV)


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def make_desc(inp):
    gp = inp["global_pos"]
    G = gp.shape[1] if gp is not None else 0
    return sc.Desc(inp["B"], inp["n"], inp["H"], inp["window"], dev_i32(inp["valid_len"]),
                   dev_i32(gp) if G > 0 else None, inp["alpha"], sc.SC_BF16 if inp["dtype"] == "bf16" else sc.SC_F32)


def run_attention(inp, band=False):
    """HIP path: window attention + score.  Returns numpy (out, lse, scores[, band scores])."""
    d = make_desc(inp)
    q, k, v = (to_dev_storage(inp[x], inp["dtype"]) for x in ("q", "k", "v"))
    out, lse, sp, bp = sc.sc_window_attention(d, q, k, v, lse=True, score_partials=True, band_probs=band)
    scores = sc.sc_ltp_score(d, sp)
    res = dict(out=out.float().cpu().numpy(), lse=lse.cpu().numpy(), scores=scores.cpu().numpy(), desc=d,
               q=q, k=k, v=v, out_t=out, scores_t=scores)
    if band:
        res["band_scores"] = sc.sc_ltp_score(d, bp, mode=sc.SC_SCORE_FROM_BAND_PROBS).cpu().numpy()
        res["band_probs"] = bp
    torch.cuda.synchronize()
    return res


def check_out(gpu, ref, dtype, what="out", bf16_step=False, count_beyond=None):
    """bf16_step: allow one bf16 step of the stored value on top (stack hidden states).  count_beyond: a
    one-element list that receives the number of elements above 2e-2 (within the step)."""
    if dtype == "f32":
        rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
        tol = 1e-4 * np.abs(ref) + 1e-6 * rms
    else:
        tol = np.full(ref.shape, 2e-2)
        if bf16_step:
            a = np.abs(ref)
            step = np.where(a > 0, np.exp2(np.floor(np.log2(np.where(a > 0, a, 1.0))) - 7), 0.0)
            tol = tol + step
    err = np.abs(gpu - ref)
    bad = err > tol
    assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance, max err {err.max():.3g}"
    if count_beyond is not None:
        count_beyond[0] += int(np.sum(err > 2e-2))
    return float(err.max()) if err.size else 0.0


def check_lse(gpu, ref, valid_len):
    B, H, n = ref.shape
    for b in range(B):
        L = int(valid_len[b])
        assert np.all(np.isneginf(gpu[b, :, L:])), "padding rows must have lse = -inf"
        r = ref[b, :, :L]
        g = gpu[b, :, :L]
        rms = float(np.sqrt(np.mean(r ** 2))) if r.size else 0.0
        err = np.abs(g - r)
        assert np.all(err <= 1e-4 * np.abs(r) + 1e-6 * rms), f"lse: max err {err.max():.3g}"


def check_scores(gpu, ref, valid_len, rel=1e-5):
    B, n = ref.shape
    worst = 0.0
    for b in range(B):
        L = int(valid_len[b])
        assert np.all(gpu[b, L:] == 0.0), "scores beyond the valid length must be 0"
        r = ref[b, :L]
        e = np.abs(gpu[b, :L] - r) / np.maximum(np.abs(r), 1e-30)
        if e.size:
            worst = max(worst, float(e.max()))
        assert np.all(e <= rel), f"scores: worst relative error {e.max():.3g}"
    return worst


def keep_sets(keep_idx, new_len):
    return [set(keep_idx[b, :new_len[b]].tolist()) for b in range(len(new_len))]


def compare_keep(gpu_keep, gpu_len, ref_scores, theta, valid_len, global_pos, keep_global=True, tag=None,
                 same_inputs=True):
    """Kept lists agree on every token whose oracle score is more than 1e-6 from theta; with
    same_inputs, a disagreement also needs |s_oracle - theta| <= 1e-5 |s_oracle| (the GPU score
    can then lie across theta).  Returns (excluded, disagreements among excluded); with a tag,
    the counts go to the run's summary."""
    excluded = disagree = 0
    s32 = ref_scores.astype(np.float32)
    for b in range(len(valid_len)):
        L = int(valid_len[b])
        g = set(int(p) for p in global_pos[b] if 0 <= p < L) if global_pos is not None else set()
        kept = set(gpu_keep[b, :gpu_len[b]].tolist())
        assert list(gpu_keep[b, :gpu_len[b]]) == sorted(kept), "kept order must be ascending"
        assert np.all(gpu_keep[b, gpu_len[b]:] == -1)
        for k in range(L):
            ref = bool(s32[b, k] > np.float32(theta)) or (keep_global and k in g)
            if abs(ref_scores[b, k] - theta) <= NEAR_THETA and not (keep_global and k in g):
                excluded += 1
                if ref != (k in kept):
                    disagree += 1
                    assert not same_inputs or abs(ref_scores[b, k] - theta) <= SCORE_REL * abs(ref_scores[b, k]), (
                        f"seq {b} token {k}: kept lists differ {abs(ref_scores[b, k] - theta):.3g} from theta, "
                        "beyond what the score tolerance allows")
                continue
            assert ref == (k in kept), f"seq {b} token {k}: oracle keep={ref}"
        assert all(k < L for k in kept)
    assert disagree <= excluded
    if tag is not None:
        record(f"{tag}: near-theta excluded {excluded} of {int(np.sum(valid_len))} tokens, disagreements {disagree}")
    return excluded, disagree
