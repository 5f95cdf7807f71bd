"""Write tests/golden/thresholds.json: the batch-wide pruning thresholds of the
single-layer workloads whose threshold is specified as a pruned fraction.

The value comes from the CPU oracle only.  Rule: sort the float32 oracle scores
of the valid, non-global tokens; among the cuts that prune between 90 % and
110 % of the target count, take the one with the widest gap between
neighbouring scores; the threshold is the float32 midpoint of that gap.  A wide
gap keeps tokens away from the threshold, where float rounding could decide.

Run:  python tests/golden/make_thresholds.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import sc_inputs as si  # noqa: E402

TARGET_PRUNED = {2: 0.30, 4: 0.50, 6: 0.30}


def gap_threshold(scores32, valid_len, global_pos, frac):
    vals = []
    for b in range(scores32.shape[0]):
        L = int(valid_len[b])
        g = set(int(p) for p in global_pos[b] if 0 <= p < L)
        vals.extend(float(scores32[b, k]) for k in range(L) if k not in g)
    v = np.sort(np.array(vals, dtype=np.float32))
    n_valid = int(np.sum(valid_len))
    target = int(round(frac * n_valid))
    lo, hi = max(1, int(0.9 * target)), min(len(v) - 1, int(1.1 * target))
    cuts = np.arange(lo, hi + 1)
    gaps = v[cuts].astype(np.float64) - v[cuts - 1].astype(np.float64)
    c = int(cuts[np.argmax(gaps)])
    theta = np.float32((np.float64(v[c - 1]) + np.float64(v[c])) / 2.0)
    return float(theta), c, float(gaps.max()), n_valid


def main():
    out = {}
    for cid, frac in TARGET_PRUNED.items():
        cfg = si.CONFIGS[cid]
        inp = si.make_attention_inputs(cfg)
        _, _, s = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                          inp["window"], inp["alpha"])
        s32 = s.astype(np.float32)
        theta, cut, gap, n_valid = gap_threshold(s32, inp["valid_len"], inp["global_pos"], frac)
        near = int(np.sum((np.abs(s - theta) <= 1e-6) & (np.arange(cfg.n)[None, :] < inp["valid_len"][:, None])))
        out[str(cid)] = dict(theta=theta, pruned=cut, valid_tokens=n_valid, target_fraction=frac, gap=gap,
                             near_threshold_1e6=near)
        print(cid, out[str(cid)])
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "thresholds.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
