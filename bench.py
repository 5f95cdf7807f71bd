#!/usr/bin/env python3
"""Benchmark of the SparseCoder hot path on one MI355X.

One step = one pass of the single-layer hot path over one batch resident in
HBM: sliding-window + global sparse attention with the exact score partials
(sc_window_attention), the importance scores (sc_ltp_score), and the
threshold / scan / compaction of the attention output (sc_ltp_prune_compact).
Default workload: batch 8, seq 4096, 12 heads x 64, bf16, window 512, 32
global tokens at seeded positions, valid lengths uniform in [2048, 4096],
threshold pruning about half of the valid tokens.

Prints one JSON line.  `value` is kept-token-layers per second (valid tokens
entering the layer, per second of GPU-stream time), from the median of the
per-step event pairs of the timed steps.

Roofline (the workload's dominant kernel, k_attn_fwd: softmax and P.V of the
window attention): its algorithmic flops (Q.K^T and P.V once per allowed
(query, key) pair and head, 4 x 64 flop) over its average launch time, measured
live with hipEvents on the launch stream, against the bf16 MFMA peak; the HBM
fraction of its algorithmic bytes alongside.  The same figures for both
window-attention launches, the HBM fractions of the score reduction and of the
prune + compaction kernels, and the VALU fraction (issue slots per pair) are
extra fields.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "kept-token-layers/sec per GPU; % MFMA (window attn) & % HBM peak (score/prune)"
HBM_PEAK_GBS = 8000.0
# VALU issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz, one non-packed op per lane per cycle (packed fp32 forms
# are not used); in Tera lane-ops per second
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# algorithmic VALU work per allowed (query, key) pair and head, in VALU issue slots: pass 1 (softmax and P.V):
# one FMA (scale, subtract the max), one exp, one add (row sum), half a max3, half a pack-convert to bf16; pass 2
# (exact probabilities for the scores): one FMA (scale, subtract the LSE), one exp, one add (column sum).  The
# exp issues at half the FMA rate (measured on gfx950: 8.2 against 4.2 cycles per wave64), so it counts twice.
VALU_SLOTS_PER_PAIR = (1 + 1 + 0.5 + 0.5) + 1 + 1 + 2 * 2
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
KERNEL_SOURCES = ("paper_2310_07109_amd/csrc/sc_attention.hip", "paper_2310_07109_amd/csrc/sc_device.h",
                  "paper_2310_07109_amd/csrc/sc_internal.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "window_attention_seq4096_traffic.json")
DOMINANT = "k_attn_fwd<1>"


# name -> (input config, workload description)
WORKLOADS = {
    "seq4096": (4, "single sparse-attention + LTP layer: B8 n4096 H12 d64 bf16, window 512, 32 seeded global "
                   "tokens, valid lengths U[2048,4096], threshold pruning ~50%"),
    "lognormal": (6, "single sparse-attention + LTP layer: B64 n1024 H12 d64 bf16, window 256, global token 0, "
                     "valid lengths round(exp(N(5.717, 0.738^2))) clipped to [1,1024] (paper-shaped), threshold "
                     "pruning ~30%"),
    "soft": ("soft", "training step of one LTP soft-pruned layer (Sec. 4.2.2 step 1): B8 n4096 H12 d64 bf16, "
                     "window 512, 32 seeded global tokens, valid lengths U[2048,4096]; forward (attention, scores, "
                     "soft mask) and backward to Q, K, V and the threshold, upstream gradients N(0,1)"),
    "encoder": ("encoder", "12-layer RoBERTa-base-shaped SparseCoder encoder: B16 n2048 D768 (12 heads x 64), "
                           "GELU feed-forward 3072, windows 64,64,128,128,256,256,512x6, global token 0, valid "
                           "lengths U[256,2048], thresholds 0.01*l/11, pruning after every layer"),
    "stack": ("stack", "12-layer attention-only encoder stack with RoBERTa-base shapes: B16 n2048 D768 (12 heads x "
                       "64), Wqkv 768x2304 and Wo 768x768 ~ N(0,0.02^2), residual + LayerNorm, no feed-forward, "
                       "window 512, global token 0, valid lengths U[256,2048], thresholds 0.01*l/11 (l = 0..11), "
                       "pruning after every layer"),
    "passes": (5, "three successive prune passes: B2 n8192 H16 d64 bf16, window 1024, 64 seeded global tokens, "
                  "full length, rank-4 amplitude-3 spike on K, thresholds 0.0005 / 0.001 / 0.002, each pass on the "
                  "previous pass's compacted Q, K, V"),
    "passes5b": ("5b", "three successive prune passes as 'passes', with the rank-4 spike on Q as well as K "
                       "(heavy-tailed scores)"),
}


def pairs_of(valid_len, global_pos, window):
    """Allowed (query, key) pairs of one layer: the window rows and the global rows."""
    pw, pg = algorithmic_counts(dict(B=len(valid_len), valid_len=valid_len, global_pos=global_pos, window=window))
    return pw + pg


def model_flops(lens_in, lens_kept, pairs, D, H, d, F):
    """FLOPs of one encoder layer broken down as the paper does (Sec. 5.1, after Electra): projections (Q, K, V
    on the layer's input tokens, the output projection on the surviving ones), sparse attention (Q.K^T and P.V
    per allowed pair and head), the feed-forward block on the surviving tokens, and other operations (softmax:
    5 per pair and head for max, subtract, exp, sum, divide; importance scores: 1 add per pair and head; two
    LayerNorms: 5 per element; GELU: 8 per hidden element).  A multiply-add counts 2."""
    t_in, t_kept = float(sum(lens_in)), float(sum(lens_kept))
    proj = 2 * t_in * D * 3 * D + 2 * t_kept * D * D
    attn = 2 * 2 * d * H * pairs
    ffn = 2 * 2 * t_kept * D * F
    other = 6 * H * pairs + 2 * 5 * t_kept * D + 8 * t_kept * F
    return dict(projection=proj, attention=attn, ffn=ffn, other=other)


# the soft-pruning backward, per allowed pair and head: five bf16 products (S = Q.K^T recomputed, dP = dO.V^T,
# dQ = dS.K, dK = dS^T.Q, dV = P^T.dO) and, in VALU issue slots, one exp (2 slots), the logit FMA, the two
# operations forming dS = P (dP + g - D) and two halves of bf16 packs (P and dS)
BWD_PRODUCTS = 5
BWD_VALU_SLOTS_PER_PAIR = 2 + 1 + 2 + 1


def measure_soft(args, sc, si, torch, np, dev="cuda:0"):
    """Times the training step of one soft-pruned layer (LTP's soft pruning): window attention with the LSE and
    score partials, scores, soft mask, and the backward to Q, K, V and the threshold."""
    cfg = si.CONFIGS[4]
    t0 = time.time()
    inp = si.make_attention_inputs(cfg)
    dy_s, dy64, dm = si.make_soft_gradients(21, cfg.B, cfg.n, cfg.H, cfg.d)
    gen_s = time.time() - t0
    B, n, H, dd = cfg.B, cfg.n, cfg.H, cfg.d

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    d = sc.Desc(B, n, H, cfg.window, i32(inp["valid_len"]), i32(inp["global_pos"]), cfg.alpha, sc.SC_BF16)
    q, k, v, dy = bf(inp["q"]), bf(inp["k"]), bf(inp["v"]), bf(dy_s)
    dmask = torch.from_numpy(dm).to(dev)
    out = torch.empty_like(q)
    lse = torch.empty((B, H, n), dtype=torch.float32, device=dev)
    sp = torch.empty(sc.sc_score_partials_size(d) // 4, dtype=torch.float32, device=dev)
    ws_attn = torch.empty(max(sc.sc_window_attention_workspace_size(d), 1), dtype=torch.uint8, device=dev)
    scores = torch.empty((B, n), dtype=torch.float32, device=dev)
    mask = torch.empty((B, n), dtype=torch.float32, device=dev)
    y = torch.empty_like(out)
    grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
             torch.empty(1, dtype=torch.float32, device=dev))
    ws_b = torch.empty(sc.sc_ltp_soft_backward_workspace_size(d), dtype=torch.uint8, device=dev)
    # threshold at the median score of the valid non-global tokens, temperature their spread
    sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, workspace=ws_attn)
    sc.sc_ltp_score(d, sp, scores=scores)
    sv = scores.cpu().numpy()
    vals = []
    for b in range(B):
        L = int(inp["valid_len"][b])
        glob = {int(x) for x in inp["global_pos"][b] if 0 <= x < L}
        vals.extend(float(sv[b, t]) for t in range(L) if t not in glob)
    theta, temp = float(np.median(vals)), max(float(np.std(vals)), 1e-6)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps)]

    def step(i):
        sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, workspace=ws_attn)
        sc.sc_ltp_score(d, sp, scores=scores)
        sc.sc_ltp_soft_mask(d, scores, theta, temp, out, mask=mask, y=y)
        if i is not None:
            ev[2 * i].record()
        sc.sc_ltp_soft_backward(d, q, k, v, out, lse, mask, temp, dy, dmask, grads=grads, workspace=ws_b)
        if i is not None:
            ev[2 * i + 1].record()

    per, mean_ms, wall_ms = timed(step, args.steps, args.warmup, torch)
    ms = median(per)
    bwd_ms = median([ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)])
    tokens = int(np.sum(inp["valid_len"]))
    pw, pg = algorithmic_counts(inp)
    pairs = H * (pw + pg)
    flops = 2.0 * dd * BWD_PRODUCTS * pairs
    # read Q, K, V, O, dY (bf16) and the LSE per valid token and head, the mask and its gradient per token; write
    # dQ, dK, dV (bf16)
    bytes_ = tokens * H * (8 * 2 * dd + 4) + tokens * 8
    t_mfma = flops / (MFMA_PEAK_TFLOPS["bf16"] * 1e12)
    t_hbm = bytes_ / (HBM_PEAK_GBS * 1e9)
    alu = BWD_VALU_SLOTS_PER_PAIR * pairs
    t_alu = alu / (VALU_PEAK_TOPS * 1e12)
    if t_mfma >= max(t_hbm, t_alu):
        roof = dict(bound="mfma", achieved=round(flops / (bwd_ms * 1e-3) / 1e12, 2), peak=MFMA_PEAK_TFLOPS["bf16"],
                    unit="TFLOP/s")
    elif t_hbm >= t_alu:
        roof = dict(bound="hbm", achieved=round(bytes_ / (bwd_ms * 1e-3) / 1e9, 1), peak=HBM_PEAK_GBS, unit="GB/s")
    else:
        roof = dict(bound="alu", achieved=round(alu / (bwd_ms * 1e-3) / 1e12, 3), peak=round(VALU_PEAK_TOPS, 2),
                    unit="T VALU lane-op/s")
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof.update(floor_mfma_us=round(t_mfma * 1e6, 2), floor_hbm_us=round(t_hbm * 1e6, 2),
                floor_alu_us=round(t_alu * 1e6, 2), traffic=None, kernel="sc_ltp_soft_backward (all its launches)",
                kernel_us=round(bwd_ms * 1e3, 2), algorithmic_flop=flops, algorithmic_bytes=bytes_)
    res = dict(ms=ms, mean_ms=mean_ms, wall_ms=wall_ms, bwd_ms=bwd_ms, tokens=tokens, theta=theta, temp=temp,
               roof=roof, gen_s=gen_s, dtheta=float(grads[3].item()))
    if not args.no_cpu_baseline:
        import oracle

        def run(rows, threads):
            sel = [inp[x][rows] for x in ("q64", "k64", "v64")]
            vl, gp = inp["valid_len"][rows], inp["global_pos"][rows]
            oracle.soft_prune_forward(*sel, vl, gp, cfg.window, cfg.alpha, theta, temp, 1, nthreads=threads)
            oracle.soft_prune_backward(*sel, vl, gp, cfg.window, cfg.alpha, theta, temp, dy64[rows],
                                       dm[rows].astype(np.float64), 1, nthreads=threads)

        n0 = int(inp["valid_len"][0])
        res["cpu_baseline"] = cpu_baseline(lambda t: run([0], t), n0, lambda t: run([0], t), n0,
                                           "token-layers/s (training step)",
                                           f"sequence 0 of the workload ({n0} tokens): soft-pruned forward and "
                                           "backward in double precision",
                                           f"the same sequence")
    return res


def measure_stack(args, sc, si, torch, np, full, dev="cuda:0"):
    """Times the 12-layer stack: sc_encoder_stack (full layers with the feed-forward block) or
    sc_encoder_attn_stack (attention-only layers)."""
    cfg = si.STACK_FULL_CONFIG if full else si.STACK_CONFIG
    t0 = time.time()
    inp = si.make_stack_inputs(cfg)
    gen_s = time.time() - t0

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    d = sc.Desc(cfg.B, cfg.n, cfg.H, cfg.window, i32(inp["valid_len"]), i32(inp["global_pos"]), cfg.alpha, sc.SC_BF16)
    x = bf(inp["x"])
    wq, wo = ([bf(w) for w in inp[k]] for k in ("wqkv", "wo"))
    th = cfg.thresholds()
    x_out = torch.empty_like(x)
    if full:
        w1, w2 = ([bf(w) for w in inp[k]] for k in ("w1", "w2"))
        ws = torch.empty(sc.sc_encoder_stack_workspace_size(d, cfg.n_layers, cfg.ffn_dim), dtype=torch.uint8,
                         device=dev)
        windows = list(inp["windows"])
    else:
        ws = torch.empty(sc.sc_encoder_attn_stack_workspace_size(d, cfg.n_layers), dtype=torch.uint8, device=dev)
        windows = [cfg.window] * cfg.n_layers
    res = {}

    def step(i):
        if full:
            res["r"] = sc.sc_encoder_stack(d, x, wq, wo, w1, w2, th, windows=windows, x_out=x_out, workspace=ws)
        else:
            res["r"] = sc.sc_encoder_attn_stack(d, x, wq, wo, th, x_out=x_out, workspace=ws)

    eager = timed(step, args.steps, args.warmup, torch)
    replayed = timed(capture(step, torch), args.steps, args.warmup, torch)
    per, mean_ms, wall_ms = replayed if args.graph else eager
    per_other = eager[0] if args.graph else replayed[0]
    # the per-layer attention times, in a second run of the same steps
    sc.sc_profile_window_kernel(True)
    timed(step, args.steps, 0, torch)
    fwd, cols = sc.sc_profile_window_kernel_read()
    sc.sc_profile_window_kernel(False)
    L = cfg.n_layers
    ms = median(per)
    kpl = res["r"][3].cpu().numpy()
    # per-layer input lengths and global positions (token 0 is global and always kept, so it stays at 0)
    lens_in = [inp["valid_len"].astype(np.int64)] + [kpl[l].astype(np.int64) for l in range(L - 1)]
    tokens = int(sum(int(np.sum(li)) for li in lens_in))
    D, F = cfg.H * cfg.d, cfg.ffn_dim
    parts = dict(projection=0.0, attention=0.0, ffn=0.0, other=0.0)
    layers = []
    for l in range(L):
        li = lens_in[l]
        gp = np.where(li[:, None] > 0, 0, -1).astype(np.int32)
        pairs = pairs_of(li, gp, windows[l])
        f = model_flops(li, kpl[l], pairs, D, cfg.H, cfg.d, F)
        for k in parts:
            parts[k] += f[k]
        layers.append(dict(tokens_in=int(np.sum(li)), kept=int(np.sum(kpl[l])), window=windows[l],
                           attn_fwd_us=round(median(fwd[l::L]) * 1e3, 2), attn_cols_us=round(median(cols[l::L]) * 1e3, 2)))
    total = sum(parts.values())
    achieved = total / (ms * 1e-3) / 1e12
    # layer 0's window attention against its own floors
    f0, b0 = attention_work(int(np.sum(lens_in[0])), cfg.H, cfg.d,
                            cfg.H * pairs_of(lens_in[0], np.where(lens_in[0][:, None] > 0, 0, -1).astype(np.int32),
                                             windows[0]))
    t0_fwd = median(fwd[0::L])
    roof = dict(bound="mfma", achieved=round(achieved, 2), peak=MFMA_PEAK_TFLOPS["bf16"], unit="TFLOP/s",
                frac=round(achieved / MFMA_PEAK_TFLOPS["bf16"], 4), traffic=None,
                kernel="whole stack step (model FLOPs as counted by model_flops)",
                layer0_attention=dict(kernel="k_attn_fwd<bf16> of layer 0", us=round(t0_fwd * 1e3, 2),
                                      mfma_frac=round(f0 / (t0_fwd * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS["bf16"], 4),
                                      hbm_frac=round(b0 / (t0_fwd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                      floor_mfma_us=round(f0 / (MFMA_PEAK_TFLOPS["bf16"] * 1e12) * 1e6, 2),
                                      floor_hbm_us=round(b0 / (HBM_PEAK_GBS * 1e9) * 1e6, 2)))
    t_in0 = float(np.sum(lens_in[0]))
    gemm0 = 2 * t_in0 * D * 3 * D + 2 * float(np.sum(kpl[0])) * D * D
    roof["layer0_gemm_floor_us"] = round(gemm0 / (MFMA_PEAK_TFLOPS["bf16"] * 1e12) * 1e6, 2)
    out = dict(ms=ms, mean_ms=mean_ms, wall_ms=wall_ms, other_ms=median(per_other), tokens=tokens,
               kept_per_layer=[int(np.sum(k)) for k in kpl],
               gen_s=gen_s, gflops={k: round(v / 1e9, 2) for k, v in parts.items()},
               total_gflops=round(total / 1e9, 2), roof=roof, layers=layers)
    if not args.no_cpu_baseline:
        import oracle
        ffn = dict(w1_list=inp["w1_64"], w2_list=inp["w2_64"]) if full else {}
        win_arg = list(inp["windows"]) if full else cfg.window

        def run_all(threads):
            oracle.encoder_stack(inp["x64"], inp["wqkv64"], inp["wo64"], inp["valid_len"], inp["global_pos"], cfg.H,
                                 win_arg, cfg.alpha, th, nthreads=threads, **ffn)

        one = [int(np.argmin(inp["valid_len"]))]

        def run_one(threads):
            oracle.encoder_stack(inp["x64"][one], inp["wqkv64"], inp["wo64"], inp["valid_len"][one],
                                 inp["global_pos"][one], cfg.H, win_arg, cfg.alpha, th, nthreads=threads, **ffn)

        units_one = None
        _, _, _, k1 = oracle.encoder_stack(inp["x64"][one], inp["wqkv64"], inp["wo64"], inp["valid_len"][one],
                                           inp["global_pos"][one], cfg.H, win_arg, cfg.alpha, th, **ffn)
        units_one = int(inp["valid_len"][one].sum()) + int(np.sum(k1[:-1]))
        out["cpu_baseline"] = cpu_baseline(run_all, tokens, run_one, units_one, "kept-token-layers/s",
                                           f"the whole workload ({cfg.B} sequences, {L} layers) in double precision",
                                           f"the shortest sequence ({int(inp['valid_len'][one].sum())} tokens), "
                                           f"{L} layers")
    return out


def kernel_source_hash():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel=DOMINANT):
    """Calibrated HBM bytes (FETCH_SIZE + WRITE_SIZE) per launch of `kernel`, from the committed counter
    measurement, if it was taken on the current kernel sources (else None)."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    c, cal = rec["counters_kib_per_dispatch"], rec["calibration"]
    try:
        return int(round(1024 * (c["FETCH_SIZE"][kernel] * cal["fetch_scale"] +
                                 c["WRITE_SIZE"][kernel] * cal["write_scale"])))
    except KeyError:
        return None


def algorithmic_counts(inp, causal=False):
    """Allowed (query, key) pairs of the non-global valid queries and of the global rows (causal: keys at or
    before the query only)."""
    import numpy as np
    r = inp["window"] // 2
    pairs_window = pairs_global = 0
    for b in range(inp["B"]):
        L = int(inp["valid_len"][b])
        g = np.array(sorted(int(p) for p in inp["global_pos"][b] if 0 <= p < L), dtype=np.int64)
        q = np.arange(L, dtype=np.int64)
        lo, hi = np.maximum(0, q - r), np.minimum(L - 1, q if causal else q + r)
        band = hi - lo + 1
        g_in = np.searchsorted(g, hi, side="right") - np.searchsorted(g, lo, side="left")
        g_reach = np.searchsorted(g, q, side="right") if causal else len(g)  # global keys the query may see
        nonglob = np.ones(L, bool)
        nonglob[g] = False
        pairs_window += int(np.sum((band + g_reach - g_in)[nonglob]))
        pairs_global += int(np.sum(g + 1)) if causal else len(g) * L
    return pairs_window, pairs_global


def median(xs):
    xs = sorted(xs)
    k = len(xs)
    return 0.0 if k == 0 else (xs[k // 2] if k % 2 else 0.5 * (xs[k // 2 - 1] + xs[k // 2]))


def attention_work(tokens, H, d, pairs):
    """Algorithmic work of one window-attention call (pairs: allowed (query, key) pairs summed over the heads):
    flops of Q.K^T and P.V once per pair; bytes of reading Q, K, V and writing O (bf16) and the LSE (fp32) per
    valid token and head."""
    return 4.0 * d * pairs, tokens * H * (4 * d * 2 + 4)


def roofline(flops, bytes_, fwd_ms, cols_ms, pairs, score=None, prune=None, traffic=None):
    """Roofline of the dominant kernel (launch 1 of the window attention) against the bf16 MFMA peak, with its
    HBM fraction; both launches against the MFMA, HBM and VALU floors; the score and prune + compaction kernels
    against HBM.  score / prune: (kernel names, microseconds, algorithmic bytes)."""
    t_mfma = flops / (MFMA_PEAK_TFLOPS["bf16"] * 1e12)
    t_hbm = bytes_ / (HBM_PEAK_GBS * 1e9)
    alu_ops = VALU_SLOTS_PER_PAIR * pairs
    t_alu = alu_ops / (VALU_PEAK_TOPS * 1e12)
    achieved = flops / (fwd_ms * 1e-3) / 1e12
    both = fwd_ms + cols_ms
    roof = dict(bound="mfma", achieved=round(achieved, 2), peak=MFMA_PEAK_TFLOPS["bf16"], unit="TFLOP/s",
                frac=round(achieved / MFMA_PEAK_TFLOPS["bf16"], 4), traffic=traffic,
                kernel="k_attn_fwd<bf16> (launch 1 of the window attention: softmax and P.V)",
                kernel_us=round(fwd_ms * 1e3, 2), algorithmic_flop=flops, algorithmic_bytes=bytes_,
                hbm_achieved_gbs=round(bytes_ / (fwd_ms * 1e-3) / 1e9, 1),
                hbm_frac=round(bytes_ / (fwd_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                floors_us=dict(mfma=round(t_mfma * 1e6, 2), hbm=round(t_hbm * 1e6, 2), valu=round(t_alu * 1e6, 2)))
    roof["window_attention_both_launches"] = dict(
        kernels="k_attn_fwd<bf16> + k_attn_cols<bf16>", us=round(both * 1e3, 2), cols_us=round(cols_ms * 1e3, 2),
        mfma_frac=round(t_mfma / (both * 1e-3), 4), hbm_frac=round(t_hbm / (both * 1e-3), 4),
        valu_frac=round(t_alu / (both * 1e-3), 4), valu_achieved_tops=round(alu_ops / (both * 1e-3) / 1e12, 3),
        valu_peak_tops=round(VALU_PEAK_TOPS, 2), valu_slots_per_pair=VALU_SLOTS_PER_PAIR)
    for key, part in (("score", score), ("prune_compact", prune)):
        if part is None:
            continue
        names, us, nbytes = part
        gbs = nbytes / (us * 1e-6) / 1e9 if us > 0 else 0.0
        roof[key] = dict(kernels=names, us=round(us, 2), algorithmic_bytes=int(nbytes), achieved_gbs=round(gbs, 1),
                         hbm_frac=round(gbs / HBM_PEAK_GBS, 4))
    return roof


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(run_all, units_all, run_one, units_one, unit, sample_all, sample_one):
    """The oracle on the host: the median of 3 runs of run_all() on every thread, then one run of run_one() on a
    single thread.  units_*: the metric's units each run processes (token-layers)."""
    import oracle
    threads = oracle.default_threads()
    times = []
    for _ in range(3):
        c0 = time.perf_counter()
        run_all(threads)
        times.append(time.perf_counter() - c0)
    t_all = median(times)
    c0 = time.perf_counter()
    run_one(1)
    t_one = time.perf_counter() - c0
    return {"value": round(units_all / t_all, 1), "unit": unit, "cores": threads, "kind": "oracle",
            "sample": f"{sample_all}; median of 3 runs on {threads} threads ({', '.join(f'{t:.2f}' for t in times)} "
                      f"s)",
            "single_thread": {"value": round(units_one / t_one, 1), "unit": unit, "cores": 1,
                              "sample": f"{sample_one}, {t_one:.2f} s"},
            "cpu_model": cpu_model(), "host_threads": os.cpu_count()}


def capture(step, torch):
    """One step recorded into a HIP graph (torch.cuda.CUDAGraph: stream capture of the library's launches; the
    library enqueues no memset, copy or synchronisation, and every buffer is preallocated).  Returns a step
    function that replays it."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(None)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(None)
    torch.cuda.synchronize()

    def replay(i):
        g.replay()
    replay.graph = g
    return replay


# Seconds of untimed load before the warmup steps of every timed run (--settle).  After idling, the GPU runs at
# a lower clock for its first few hundred milliseconds of load: the seq-4096 step measured 0.155-0.160 ms per step
# after 5 or 10 warmup steps and 0.141-0.143 ms after 3000 (0.5 s), in one process, and fell back to 0.160 after
# a 2-second pause.
SETTLE_S = 0.5
TWO_STREAMS = None  # created first thing in main (see there)


def timed(step, steps, warmup, torch):
    """Runs the step untimed for SETTLE_S seconds and `warmup` times, then `steps` timed ones bracketed by
    synchronisations, with an event on the launch stream before every step and after the last.  step(i) gets
    the step index (None when untimed).  Returns (per-step milliseconds, mean milliseconds over the bracket,
    wall milliseconds per step)."""
    t_end = time.perf_counter() + SETTLE_S
    while time.perf_counter() < t_end:
        for _ in range(8):
            step(None)
        torch.cuda.synchronize()
    for _ in range(warmup):
        step(None)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    w0 = time.perf_counter()
    for i in range(steps):
        ev[i].record()
        step(i)
    ev[steps].record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - w0) * 1e3 / max(steps, 1)
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return per, ev[0].elapsed_time(ev[steps]) / max(steps, 1), wall


def measure(sc, si, torch, np, inp, theta, steps, warmup, dev="cuda:0", keep_ratio=None, causal=False,
            band=False, graph=True):
    """Times `steps` steps (window attention with score partials, scores, prune + compaction of O) after
    `warmup` untimed ones.  theta None picks the median score of the valid non-global tokens (about half
    pruned), from one untimed step.  keep_ratio: prune by the top-k rule (sc_topk_prune_compact) instead of
    the threshold.  causal: the causal variant of the attention.  band: the paper's score path (Sec. 5.5):
    the window attention stores every probability in the band layout and the scores are summed from it."""
    B, n, H, dd, G = inp["B"], inp["n"], inp["H"], inp["d"], inp["G"]

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    d = sc.Desc(B, n, H, inp["window"], i32(inp["valid_len"]), i32(inp["global_pos"]), inp["alpha"], sc.SC_BF16,
                causal=causal)
    q, k, v = bf(inp["q"]), bf(inp["k"]), bf(inp["v"])
    out = torch.empty_like(q)
    lse = torch.empty((B, H, n), dtype=torch.float32, device=dev)
    sp = torch.empty(sc.sc_score_partials_size(d) // 4, dtype=torch.float32, device=dev)
    bp = torch.empty(sc.sc_band_probs_size(d) // 4, dtype=torch.float32, device=dev) if band else None
    ws_score = torch.empty(max(sc.sc_ltp_score_workspace_size(d, sc.SC_SCORE_FROM_BAND_PROBS), 1),
                           dtype=torch.uint8, device=dev) if band else None
    ws_attn = torch.empty(max(sc.sc_window_attention_workspace_size(d), 1), dtype=torch.uint8, device=dev)
    scores = torch.empty((B, n), dtype=torch.float32, device=dev)
    oc = torch.empty_like(out)
    outs = dict(keep_idx=torch.empty((B, n), dtype=torch.int32, device=dev),
                new_len=torch.empty((B,), dtype=torch.int32, device=dev),
                new_global_pos=torch.empty((B, max(G, 1)), dtype=torch.int32, device=dev),
                orig_idx_out=torch.empty((B, n), dtype=torch.int32, device=dev))
    ws_prune = torch.empty(sc.sc_ltp_prune_compact_workspace_size(d), dtype=torch.uint8, device=dev)
    if theta is None and keep_ratio is None:
        sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, workspace=ws_attn)
        sc.sc_ltp_score(d, sp, scores=scores)
        sv = scores.cpu().numpy()
        vals = []
        for b in range(B):
            L = int(inp["valid_len"][b])
            glob = {int(x) for x in inp["global_pos"][b] if 0 <= x < L}
            vals.extend(float(sv[b, t]) for t in range(L) if t not in glob)
        theta = float(np.median(vals)) if vals else 0.0
    sev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    marks = [False]

    def step(i):
        mark = marks[0] and i is not None
        if band:
            sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=None, band_probs=bp,
                                   workspace=ws_attn)
        else:
            sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, workspace=ws_attn)
        if mark:
            sev[i][0].record()
        if band:
            sc.sc_ltp_score(d, bp, mode=sc.SC_SCORE_FROM_BAND_PROBS, scores=scores, workspace=ws_score)
        else:
            sc.sc_ltp_score(d, sp, scores=scores)
        if mark:
            sev[i][1].record()
        if keep_ratio is None:
            sc.sc_ltp_prune_compact(d, scores, theta, True, [out], dsts=[oc], outs=outs, workspace=ws_prune)
        else:
            sc.sc_topk_prune_compact(d, scores, keep_ratio, True, [out], dsts=[oc], outs=outs, workspace=ws_prune)
        if mark:
            sev[i][2].record()

    # the headline: steps bracketed by one event each, launched eagerly or (graph) replayed from a HIP graph;
    # the other mode is timed too
    eager = timed(step, steps, warmup, torch)
    replayed = timed(capture(step, torch), steps, warmup, torch)
    per, mean_ms, wall_ms = replayed if graph else eager
    per_other = eager[0] if graph else replayed[0]
    # the breakdown, in a second run of the same steps: the window attention's two launches (the library's
    # events) and the score and prune + compaction calls (events between the calls)
    sc.sc_profile_window_kernel(True)
    marks[0] = True
    timed(step, steps, 0, torch)
    fwd, cols = sc.sc_profile_window_kernel_read()
    sc.sc_profile_window_kernel(False)
    score_us = median([sev[i][0].elapsed_time(sev[i][1]) for i in range(steps)]) * 1e3
    prune_us = median([sev[i][1].elapsed_time(sev[i][2]) for i in range(steps)]) * 1e3

    tokens = int(np.sum(inp["valid_len"]))
    kept = outs["new_len"].cpu().tolist()
    pairs_w, pairs_g = algorithmic_counts(inp, causal)
    pairs = H * (pairs_w + pairs_g)
    flops, bytes_ = attention_work(tokens, H, dd, pairs)
    # score reduction: read the partials, write the scores; prune + compaction: read the scores, write the kept
    # indices, composed indices and lengths, read and write each kept row of O
    score_bytes = sp.numel() * 4 + 4 * B * n
    score_kernels = "k_score_from_partials"
    if band:  # the paper's layout: read each valid token's band and global-column entries and the global rows
        r = inp["window"] // 2
        g_used = sum(len([p for p in inp["global_pos"][b] if 0 <= p < inp["valid_len"][b]]) for b in range(B))
        score_bytes = 4 * H * (tokens * (min(2 * r + 1, n)) + 2 * g_used * n) + 4 * B * n
        score_kernels = "k_band_rows + k_band_keys + k_score_from_partials"
    prune_bytes = 4 * B * n * 3 + 2 * sum(kept) * H * dd * 2
    roof = roofline(flops, bytes_, median(fwd), median(cols), pairs,
                    score=(score_kernels, score_us, score_bytes),
                    prune=("k_prune_compact" if keep_ratio is None else "k_prune_scan + k_gather_rows", prune_us,
                           prune_bytes))
    return dict(ms=median(per), mean_ms=mean_ms, wall_ms=wall_ms, fwd_ms=median(fwd), cols_ms=median(cols),
                tokens=tokens, kept=kept, flops=flops, bytes=bytes_, roof=roof, theta=theta, pairs=pairs,
                other_ms=median(per_other))


def two_streams(sc, torch, np, inp, theta, steps, warmup, dev="cuda:0", causal=False):
    """The same step with the batch's sequences split into two halves (even and odd indices), each half's
    window attention, scores and prune + compaction enqueued on a stream of its own (default priority), the
    halves alternating.  Results are identical to the single call's; the halves' kernels overlap each other's
    launch tails.  Returns milliseconds per step of the whole batch, between an event before the first step
    (both streams wait on it) and one after both streams' last."""
    B, n, H, G = inp["B"], inp["n"], inp["H"], inp["G"]

    def half(rows):
        sel = np.array(rows)
        d = sc.Desc(len(rows), n, H, inp["window"],
                    torch.from_numpy(np.ascontiguousarray(inp["valid_len"][sel], dtype=np.int32)).to(dev),
                    torch.from_numpy(np.ascontiguousarray(inp["global_pos"][sel], dtype=np.int32)).to(dev),
                    inp["alpha"], sc.SC_BF16, causal=causal)
        t = dict(d=d)
        for x in ("q", "k", "v"):
            t[x] = torch.from_numpy(np.ascontiguousarray(inp[x][sel]).view(np.int16)).to(dev).view(torch.bfloat16)
        t["out"], t["oc"] = torch.empty_like(t["q"]), torch.empty_like(t["q"])
        t["lse"] = torch.empty((len(rows), H, n), dtype=torch.float32, device=dev)
        t["sp"] = torch.empty(sc.sc_score_partials_size(d) // 4, dtype=torch.float32, device=dev)
        t["ws_attn"] = torch.empty(max(sc.sc_window_attention_workspace_size(d), 1), dtype=torch.uint8, device=dev)
        t["scores"] = torch.empty((len(rows), n), dtype=torch.float32, device=dev)
        t["outs"] = dict(keep_idx=torch.empty((len(rows), n), dtype=torch.int32, device=dev),
                         new_len=torch.empty((len(rows),), dtype=torch.int32, device=dev),
                         new_global_pos=torch.empty((len(rows), max(G, 1)), dtype=torch.int32, device=dev),
                         orig_idx_out=torch.empty((len(rows), n), dtype=torch.int32, device=dev))
        t["ws_prune"] = torch.empty(sc.sc_ltp_prune_compact_workspace_size(d), dtype=torch.uint8, device=dev)
        return t

    halves = [half(list(range(0, B, 2))), half(list(range(1, B, 2)))]
    streams = TWO_STREAMS or [torch.cuda.Stream(), torch.cuda.Stream()]
    for t, st in zip(halves, streams):
        t["stream"] = st

    def run(t):
        d, st = t["d"], t["stream"]
        sc.sc_window_attention(d, t["q"], t["k"], t["v"], out=t["out"], lse=t["lse"], score_partials=t["sp"],
                               workspace=t["ws_attn"], stream=st)
        sc.sc_ltp_score(d, t["sp"], scores=t["scores"], stream=st)
        sc.sc_ltp_prune_compact(d, t["scores"], theta, True, [t["out"]], dsts=[t["oc"]], outs=t["outs"],
                                workspace=t["ws_prune"], stream=st)

    def step():
        for t in halves:
            run(t)

    t_end = time.perf_counter() + SETTLE_S
    while time.perf_counter() < t_end:
        for _ in range(8):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    main = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(main)
    for t in halves:
        t["stream"].wait_event(e0)
    for _ in range(steps):
        step()
    for t in halves:
        e = torch.cuda.Event()
        e.record(t["stream"])
        main.wait_event(e)
    e1.record(main)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - w0) * 1e3 / max(steps, 1)
    return e0.elapsed_time(e1) / max(steps, 1), wall


def measure_passes(sc, si, torch, np, cfg, steps, warmup, dev="cuda:0", graph=True):
    """Times `steps` steps of three successive prune passes: each pass runs the window attention with score
    partials, the scores, and the threshold prune + compaction of Q, K and V into the next pass's buffers, with
    the lengths and global positions staying on the device."""
    inp = si.make_attention_inputs(cfg)
    B, n, H, dd, G = cfg.B, cfg.n, cfg.H, cfg.d, cfg.n_global

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    P = len(cfg.thresholds)
    qkv = [[bf(inp["q"]), bf(inp["k"]), bf(inp["v"])]] + [[torch.empty((B, n, H, dd), dtype=torch.bfloat16,
                                                                       device=dev) for _ in range(3)]
                                                          for _ in range(P)]
    lens = [i32(inp["valid_len"])] + [torch.empty((B,), dtype=torch.int32, device=dev) for _ in range(P)]
    gps = [i32(inp["global_pos"])] + [torch.empty((B, G), dtype=torch.int32, device=dev) for _ in range(P)]
    descs = [sc.Desc(B, n, H, cfg.window, lens[p], gps[p], cfg.alpha, sc.SC_BF16) for p in range(P)]
    d0 = descs[0]
    out = torch.empty_like(qkv[0][0])
    lse = torch.empty((B, H, n), dtype=torch.float32, device=dev)
    sp = torch.empty(sc.sc_score_partials_size(d0) // 4, dtype=torch.float32, device=dev)
    ws_attn = torch.empty(max(sc.sc_window_attention_workspace_size(d0), 1), dtype=torch.uint8, device=dev)
    scores = torch.empty((B, n), dtype=torch.float32, device=dev)
    ws_prune = torch.empty(sc.sc_ltp_prune_compact_workspace_size(d0), dtype=torch.uint8, device=dev)
    keep = torch.empty((B, n), dtype=torch.int32, device=dev)

    def step(i):
        for p in range(P):
            d = descs[p]
            sc.sc_window_attention(d, *qkv[p], out=out, lse=lse, score_partials=sp, workspace=ws_attn)
            sc.sc_ltp_score(d, sp, scores=scores)
            sc.sc_ltp_prune_compact(d, scores, cfg.thresholds[p], True, qkv[p], dsts=qkv[p + 1], want_orig=False,
                                    outs=dict(keep_idx=keep, new_len=lens[p + 1], new_global_pos=gps[p + 1]),
                                    workspace=ws_prune)

    eager = timed(step, steps, warmup, torch)
    replayed = timed(capture(step, torch), steps, warmup, torch)
    per, mean_ms, wall_ms = replayed if graph else eager
    per_other = eager[0] if graph else replayed[0]
    # the per-pass attention times, in a second run of the same steps
    sc.sc_profile_window_kernel(True)
    timed(step, steps, 0, torch)
    fwd, cols = sc.sc_profile_window_kernel_read()
    sc.sc_profile_window_kernel(False)
    lens_h = [inp["valid_len"].astype(np.int64)] + [lens[p + 1].cpu().numpy().astype(np.int64) for p in range(P)]
    gps_h = [inp["global_pos"]] + [gps[p + 1].cpu().numpy() for p in range(P)]
    tokens = int(sum(int(np.sum(lens_h[p])) for p in range(P)))
    # the dominant kernel is pass 1's launch 1
    pw, pg = algorithmic_counts(dict(B=B, valid_len=lens_h[0], global_pos=gps_h[0], window=cfg.window))
    flops, bytes_ = attention_work(int(np.sum(lens_h[0])), H, dd, H * (pw + pg))
    roof = roofline(flops, bytes_, median(fwd[0::P]), median(cols[0::P]), H * (pw + pg))
    roof["kernel"] = "k_attn_fwd<bf16> of pass 1 (launch 1 of the window attention: softmax and P.V)"
    roof["traffic"] = None
    passes = []
    for p in range(P):
        pw_, pg_ = algorithmic_counts(dict(B=B, valid_len=lens_h[p], global_pos=gps_h[p], window=cfg.window))
        passes.append(dict(tokens_in=lens_h[p].tolist(), kept=lens_h[p + 1].tolist(), allowed_pairs=H * (pw_ + pg_),
                           attn_fwd_us=round(median(fwd[p::P]) * 1e3, 2),
                           attn_cols_us=round(median(cols[p::P]) * 1e3, 2)))
    return dict(ms=median(per), mean_ms=mean_ms, wall_ms=wall_ms, tokens=tokens, roof=roof, passes=passes, inp=inp,
                lens=lens_h, gps=gps_h, other_ms=median(per_other))


def probe_valu():
    """Issue rate of v_fma_f32 and v_exp_f32 per SIMD: 2048 workgroups (8 waves per SIMD on 256 CUs), each
    thread 8 independent chains, so that the time is set by issue, not latency.  Cycles at the 2.4 GHz peak
    clock; the ratio does not depend on the clock."""
    import ctypes
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2310_07109_amd", "libsc_probe.so")
    lib = ctypes.CDLL(path)
    lib.sc_probe_valu_rate.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double)]
    simds, clock = 256 * 4, 2.4e9
    res = {}
    for op, name in ((0, "v_fma_f32"), (1, "v_exp_f32")):
        runs = []
        for _ in range(3):
            ms, wi = ctypes.c_double(), ctypes.c_double()
            rc = lib.sc_probe_valu_rate(op, 2048, 2048, ctypes.byref(ms), ctypes.byref(wi))
            if rc != 0:
                raise RuntimeError(f"probe failed: {rc}")
            runs.append(ms.value * 1e-3 * clock * simds / wi.value)
        res[name] = round(median(runs), 3)
    print(json.dumps({"probe": "VALU issue rate per SIMD (wave64 instructions)", "cycles_per_instruction": res,
                      "exp_over_fma": round(res["v_exp_f32"] / res["v_fma_f32"], 3), "clock_ghz": clock / 1e9,
                      "setup": "2048 workgroups x 256 threads (8 waves per SIMD), 8 independent chains per thread, "
                               "65536 instructions per thread, median of 3 timed launches"}))


def probe_lds():
    """LDS read throughput per CU of ds_read_b128 and ds_read_b64_tr_b16: 1024 workgroups (4 of 4 waves per CU on
    256 CUs, the window attention's residency), 32 KB of LDS each, groups of 8 independent reads.  Bytes per
    cycle at the 2.4 GHz peak clock."""
    import ctypes
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2310_07109_amd", "libsc_probe.so")
    lib = ctypes.CDLL(path)
    lib.sc_probe_lds_rate.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_double)]
    cus, clock = 256, 2.4e9
    res = {}
    for op, name in ((0, "ds_read_b128"), (1, "ds_read_b64_tr_b16")):
        runs = []
        for _ in range(3):
            ms, nb = ctypes.c_double(), ctypes.c_double()
            rc = lib.sc_probe_lds_rate(op, 1024, 4096, ctypes.byref(ms), ctypes.byref(nb))
            if rc != 0:
                raise RuntimeError(f"probe failed: {rc}")
            runs.append(nb.value / cus / (ms.value * 1e-3 * clock))
        res[name] = round(median(runs), 1)
    print(json.dumps({"probe": "LDS read throughput per CU (bytes per cycle)", "bytes_per_cycle": res,
                      "tr_over_b128": round(res["ds_read_b64_tr_b16"] / res["ds_read_b128"], 3),
                      "clock_ghz": clock / 1e9,
                      "setup": "1024 workgroups x 256 threads (4 per CU), 32 KB LDS each, groups of 8 independent "
                               "reads, 4096 groups per thread, median of 3 timed launches"}))


def sweep(args, sc, si, torch, np):
    """Window and length sweeps of the same step (one JSON line per point).  Window sweep: B8 n4096;
    length sweep: window 512 and B = 32768 / n padded tokens; both H12 bf16, 32 global tokens, valid lengths
    U[n/2, n], the threshold at the median score (about half pruned)."""
    base = si.CONFIGS[4]
    points = [("window", 4096, w) for w in (16, 64, 128, 256, 512, 1024)]
    points += [("length", n, 512) for n in (1024, 2048, 4096, 8192, 16384)]
    for kind, n, w in points:
        B = 8 if kind == "window" else 32768 // n
        inp = si.make_attention_inputs(base, B=B, n=n, window=w, len_range=(n // 2, n))
        m = measure(sc, si, torch, np, inp, None, args.steps, args.warmup, graph=args.graph)
        print(json.dumps({
            "sweep": kind, "n": n, "window": w, "batch": B, "valid_tokens": m["tokens"],
            "allowed_pairs": m["pairs"], "ms_per_step": round(m["ms"], 4),
            "value": round(m["tokens"] / (m["ms"] * 1e-3), 1), "unit": "kept-token-layers/s",
            "attention_us": round((m["fwd_ms"] + m["cols_ms"]) * 1e3, 2),
            "ns_per_pair": round((m["fwd_ms"] + m["cols_ms"]) * 1e6 / m["pairs"], 4),
            "roofline": m["roof"], "kept_fraction": round(sum(m["kept"]) / m["tokens"], 3)}), flush=True)


def main():
    global SETTLE_S, TWO_STREAMS
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle", type=float, default=SETTLE_S, metavar="SECONDS",
                    help="untimed load before each timed run's warmup steps, so that the GPU runs at its sustained "
                         "clock (0: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-two-streams", action="store_true",
                    help="skip the extra measurement of the batch as two halves on two streams (kernel traces: it "
                         "overlaps kernels)")
    ap.add_argument("--graph", action="store_true",
                    help="time steps replayed from a HIP graph captured once (default: eager launches; the other "
                         "mode's time is reported beside it either way)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the run, copy MIB MiB once on the GPU (a reference kernel of known traffic for "
                         "hardware counters)")
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="seq4096",
                    help="seq4096: B8 n4096 window 512, 32 global tokens (the headline line); lognormal: B64 n1024 "
                         "window 256, one global token, paper-shaped lognormal lengths; stack: the 12-layer "
                         "attention-only stack, B16 n2048; encoder: the 12-layer stack with feed-forward blocks; "
                         "passes / passes5b: three successive prune passes at B2 n8192 window 1024; soft: training "
                         "step (forward and backward) of one soft-pruned layer at seq4096")
    ap.add_argument("--prune", choices=("threshold", "topk"), default="threshold",
                    help="pruning rule of the step: the layer threshold (the paper's rule) or top-k by keep ratio")
    ap.add_argument("--keep-ratio", type=float, default=0.5, help="top-k rule: fraction of candidates kept")
    ap.add_argument("--causal", action="store_true",
                    help="the causal variant of the attention (keys after the query never attended); the "
                         "threshold is then the median score (the stored one belongs to the bidirectional scores)")
    ap.add_argument("--score", choices=("partials", "band"), default="partials",
                    help="partials: the fused column-sum partials (default); band: the paper's score path, every "
                         "probability stored in the band layout and summed from it (Sec. 5.5)")
    ap.add_argument("--probe-valu", action="store_true",
                    help="instead of the step, measure the SIMD issue rate of v_fma_f32 and v_exp_f32 (the two VALU "
                         "forms the window attention's VALU floor counts), one JSON line")
    ap.add_argument("--probe-lds", action="store_true",
                    help="measure the LDS read throughput of the attention's fragment reads and exit")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the single measurement, sweep the window (n 4096) and the length (window "
                         "512), one JSON line per point")
    args = ap.parse_args()
    SETTLE_S = max(args.settle, 0.0)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the hot path runs on a single MI355X; --gpus {args.gpus} is not "
              "supported (sharding across GPUs is described, not built).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2310_07109_amd as sc
    import sc_inputs as si

    torch.cuda.set_device(0)
    # the two-stream measurement's streams, created and given work before anything else runs: a stream takes
    # one of the device's hardware queues at its first work, and two streams first used late in the run (after
    # the single-stream measurement) ran one after the other, as if on one queue (0.170 against 0.122 ms per
    # step)
    TWO_STREAMS = [torch.cuda.Stream(), torch.cuda.Stream()]
    for st in TWO_STREAMS:
        with torch.cuda.stream(st):
            torch.zeros(1, device="cuda:0")
    torch.cuda.synchronize()
    dev = "cuda:0"
    if args.probe_valu:
        probe_valu()
        return
    if args.probe_lds:
        probe_lds()
        return
    if args.sweep:
        sweep(args, sc, si, torch, np)
        return
    cid, desc = WORKLOADS[args.workload]
    common = {"n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "settle_s": SETTLE_S, "higher_is_better": True,
              "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic"}
    launch = "HIP graph replay (one capture of the step)" if args.graph else "eager launches"
    if cid == "soft":
        m = measure_soft(args, sc, si, torch, np, dev)
        line = {
            "metric": METRIC, "value": round(m["tokens"] / (m["ms"] * 1e-3), 1),
            "unit": "token-layers/s (training step)", **common, "ms_per_step": round(m["ms"], 4),
            "mean_ms_per_step": round(m["mean_ms"], 4),
            "config": {"workload": desc, "valid_tokens": m["tokens"], "threshold": m["theta"],
                       "temperature": m["temp"], "parallelism": "none (1 GPU)"},
            "roofline": m["roof"], "backward_ms": round(m["bwd_ms"], 4), "dtheta": m["dtheta"],
            "input_generation_s": round(m["gen_s"], 1)}
        if "cpu_baseline" in m:
            line["cpu_baseline"] = m["cpu_baseline"]
        print(json.dumps(line), flush=True)
        return
    if cid in ("encoder", "stack"):
        m = measure_stack(args, sc, si, torch, np, full=cid == "encoder", dev=dev)
        line = {
            "metric": METRIC, "value": round(m["tokens"] / (m["ms"] * 1e-3), 1), "unit": "kept-token-layers/s",
            **common, "ms_per_step": round(m["ms"], 4), "mean_ms_per_step": round(m["mean_ms"], 4),
            ("eager_ms_per_step" if args.graph else "graph_replay_ms_per_step"): round(m["other_ms"], 4),
            "config": {"workload": desc, "layer_input_tokens": m["tokens"], "kept_per_layer": m["kept_per_layer"],
                       "launch": launch, "parallelism": "none (1 GPU)"},
            "model_gflops": m["gflops"], "model_gflops_total": m["total_gflops"], "roofline": m["roof"],
            "layers": m["layers"], "input_generation_s": round(m["gen_s"], 1)}
        if "cpu_baseline" in m:
            line["cpu_baseline"] = m["cpu_baseline"]
        print(json.dumps(line), flush=True)
        return
    if args.workload.startswith("passes"):
        cfg = si.CONFIGS[cid]
        t0 = time.time()
        m = measure_passes(sc, si, torch, np, cfg, args.steps, args.warmup, dev, graph=args.graph)
        gen_s = time.time() - t0
        line = {
            "metric": METRIC, "value": round(m["tokens"] / (m["ms"] * 1e-3), 1), "unit": "kept-token-layers/s",
            **common, "ms_per_step": round(m["ms"], 4), "mean_ms_per_step": round(m["mean_ms"], 4),
            "config": {"workload": desc, "batch": cfg.B, "seq_len": cfg.n, "heads": cfg.H, "head_dim": cfg.d,
                       "window": cfg.window, "global_tokens": cfg.n_global, "thresholds": cfg.thresholds,
                       "pass_input_tokens": m["tokens"], "launch": launch, "parallelism": "none (1 GPU)"},
            ("eager_ms_per_step" if args.graph else "graph_replay_ms_per_step"): round(m["other_ms"], 4),
            "roofline": m["roof"], "passes": m["passes"], "setup_s": round(gen_s, 1)}
        if not args.no_cpu_baseline:
            import oracle
            inp = m["inp"]

            def run(rows, threads):
                q64, k64, v64 = (inp[x][rows] for x in ("q64", "k64", "v64"))
                vl, gp = inp["valid_len"][rows].copy(), inp["global_pos"][rows].copy()
                for theta in cfg.thresholds:
                    _, _, rs = oracle.sparse_attention(q64, k64, v64, vl, gp, cfg.window, cfg.alpha, nthreads=threads)
                    rk, rnl, rngp, _ = oracle.ltp_prune(rs.astype(np.float32), vl, gp, theta, 1)
                    q2, k2, v2 = (np.zeros_like(x) for x in (q64, k64, v64))
                    for b in range(len(rows)):
                        idx = rk[b, :rnl[b]]
                        q2[b, :len(idx)], k2[b, :len(idx)], v2[b, :len(idx)] = q64[b, idx], k64[b, idx], v64[b, idx]
                    q64, k64, v64, vl, gp = q2, k2, v2, rnl.astype(np.int32), rngp

            one = int(m["lens"][0][0]) + sum(int(m["lens"][p][0]) for p in range(1, len(cfg.thresholds)))
            line["cpu_baseline"] = cpu_baseline(lambda t: run(list(range(cfg.B)), t), m["tokens"],
                                                lambda t: run([0], t), one, "kept-token-layers/s",
                                                f"the whole workload ({cfg.B} sequences, three passes) in double "
                                                "precision", "sequence 0, three passes")
        print(json.dumps(line), flush=True)
        return
    cfg = si.CONFIGS[cid]
    with open(os.path.join(ROOT, "tests", "golden", "thresholds.json")) as f:
        theta = json.load(f)[str(cid)]["theta"]
    t0 = time.time()
    inp = si.make_attention_inputs(cfg)
    gen_s = time.time() - t0
    keep_ratio = args.keep_ratio if args.prune == "topk" else None
    if args.causal:
        theta = None
    m = measure(sc, si, torch, np, inp, theta, args.steps, args.warmup, dev, keep_ratio=keep_ratio,
                causal=args.causal, band=args.score == "band", graph=args.graph)
    theta = m["theta"]
    ms, tokens = m["ms"], m["tokens"]
    roof = m["roof"]
    # the recorded counters belong to the (bidirectional, threshold-pruned) seq4096 workload
    roof["traffic"] = recorded_traffic() if (args.workload == "seq4096" and not args.causal and
                                             keep_ratio is None and args.score == "partials") else None
    value = tokens / (ms * 1e-3)
    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "kept-token-layers/s", **common,
        "ms_per_step": round(ms, 4), "mean_ms_per_step": round(m["mean_ms"], 4),
        "config": {"workload": desc,
                   "batch": cfg.B, "seq_len": cfg.n, "heads": cfg.H, "head_dim": cfg.d, "window": cfg.window,
                   "global_tokens": cfg.n_global, "valid_tokens": tokens,
                   "pruning": (f"top-k, keep ratio {keep_ratio}" if keep_ratio is not None else
                               f"threshold {theta}"), "attention": "causal" if args.causal else "bidirectional",
                   "scores": "band layout (paper)" if args.score == "band" else "fused column-sum partials",
                   "launch": launch, "parallelism": "none (1 GPU)"},
        ("eager_ms_per_step" if args.graph else "graph_replay_ms_per_step"): round(m["other_ms"], 4),
        "roofline": roof,
        "kept_per_sequence": m["kept"],
        "wall_ms_per_step": round(m["wall_ms"], 4),
    }
    if args.workload == "seq4096" and args.score == "partials" and keep_ratio is None and not args.no_two_streams:
        ms2, wall2 = two_streams(sc, torch, np, inp, theta, args.steps, args.warmup, dev, causal=args.causal)
        result["two_streams"] = {"ms_per_step": round(ms2, 4), "wall_ms_per_step": round(wall2, 4),
                                 "value": round(tokens / (ms2 * 1e-3), 1),
                                 "unit": "kept-token-layers/s",
                                 "how": "the same 8 sequences as two halves (even and odd indices), each half's three "
                                        "calls on a stream of its own; not the headline"}
    if not args.no_cpu_baseline:
        import oracle

        def run(rows, threads):
            _, _, rs = oracle.sparse_attention(inp["q64"][rows], inp["k64"][rows], inp["v64"][rows],
                                               inp["valid_len"][rows], inp["global_pos"][rows], cfg.window, cfg.alpha,
                                               nthreads=threads, causal=args.causal)
            if keep_ratio is None:
                oracle.ltp_prune(rs.astype(np.float32), inp["valid_len"][rows], inp["global_pos"][rows], theta, 1)
            else:
                oracle.topk_prune(rs.astype(np.float32), inp["valid_len"][rows], inp["global_pos"][rows], keep_ratio,
                                  1)

        allrows = list(range(cfg.B))
        result["cpu_baseline"] = cpu_baseline(lambda t: run(allrows, t), tokens, lambda t: run([0], t),
                                              int(inp["valid_len"][0]), "kept-token-layers/s",
                                              f"the whole workload ({cfg.B} sequences, one layer: attention, scores, "
                                              "pruning) in double precision",
                                              f"sequence 0 ({int(inp['valid_len'][0])} tokens), one layer")
    result["input_generation_s"] = round(gen_s, 1)
    if args.copy_calibration > 0:
        nb = args.copy_calibration << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = nb
    print(json.dumps(result), flush=True)

if __name__ == "__main__":
    main()
