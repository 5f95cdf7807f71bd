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
entering the layer, per second of wall time on the GPU stream).
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
    "encoder": (None, "12-layer RoBERTa-base-shaped SparseCoder encoder: B16 n2048 D768 (12 heads x 64), GELU "
                      "feed-forward 3072, windows 64,64,128,128,256,256,512x6, global token 0, valid lengths "
                      "U[256,2048], thresholds 0.01*l/11, pruning after every layer"),
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

    def step(i=None):
        sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, workspace=ws_attn)
        sc.sc_ltp_score(d, sp, scores=scores)
        sc.sc_ltp_soft_mask(d, scores, theta, temp, out, mask=mask, y=y)
        if i is not None:
            ev[2 * i].record()
        sc.sc_ltp_soft_backward(d, q, k, v, out, lse, mask, temp, dy, dmask, grads=grads, workspace=ws_b)
        if i is not None:
            ev[2 * i + 1].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    bwd_ms = sum(ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)) / args.steps
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
    res = dict(ms=ms, bwd_ms=bwd_ms, tokens=tokens, theta=theta, temp=temp, roof=roof, gen_s=gen_s,
               dtheta=float(grads[3].item()))
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.default_threads()
        c0 = time.perf_counter()
        rows = [0]
        sel = [inp[x][rows] for x in ("q64", "k64", "v64")]
        vl, gp = inp["valid_len"][rows], inp["global_pos"][rows]
        oracle.soft_prune_forward(*sel, vl, gp, cfg.window, cfg.alpha, theta, temp, 1, nthreads=threads)
        oracle.soft_prune_backward(*sel, vl, gp, cfg.window, cfg.alpha, theta, temp, dy64[rows],
                                   dm[rows].astype(np.float64), 1, nthreads=threads)
        cpu_s = time.perf_counter() - c0
        res["cpu_baseline"] = {"value": round(int(vl.sum()) / cpu_s, 1), "unit": "token-layers/s (training step)",
                               "cores": threads, "kind": "oracle",
                               "sample": f"sequence 0 of the workload ({int(vl.sum())} tokens): soft-pruned "
                                         f"forward and backward in double precision, {cpu_s:.2f} s"}
    return res


def measure_encoder(args, sc, si, torch, np, dev="cuda:0"):
    """Times the full encoder stack (sc_encoder_stack over 12 layers)."""
    cfg = si.STACK_FULL_CONFIG
    t0 = time.time()
    inp = si.make_stack_inputs(cfg)
    gen_s = time.time() - t0

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    d = sc.Desc(cfg.B, cfg.n, cfg.H, cfg.window, i32(inp["valid_len"]), i32(inp["global_pos"]), cfg.alpha, sc.SC_BF16)
    x = bf(inp["x"])
    wq, wo, w1, w2 = ([bf(w) for w in inp[k]] for k in ("wqkv", "wo", "w1", "w2"))
    th = cfg.thresholds()
    ws = torch.empty(sc.sc_encoder_stack_workspace_size(d, cfg.n_layers, cfg.ffn_dim), dtype=torch.uint8, device=dev)
    x_out = torch.empty_like(x)

    def step():
        return sc.sc_encoder_stack(d, x, wq, wo, w1, w2, th, windows=inp["windows"], x_out=x_out, workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        res = step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    kpl = res[3].cpu().numpy()
    # per-layer input lengths and global positions (token 0 is global and always kept, so it stays at 0)
    lens_in = [inp["valid_len"].astype(np.int64)] + [kpl[l].astype(np.int64) for l in range(cfg.n_layers - 1)]
    tokens = int(sum(int(np.sum(li)) for li in lens_in))
    D, F = cfg.H * cfg.d, cfg.ffn_dim
    parts = dict(projection=0.0, attention=0.0, ffn=0.0, other=0.0)
    for l in range(cfg.n_layers):
        li = lens_in[l]
        gp = np.where(li[:, None] > 0, 0, -1).astype(np.int32)
        f = model_flops(li, kpl[l], pairs_of(li, gp, inp["windows"][l]), D, cfg.H, cfg.d, F)
        for k in parts:
            parts[k] += f[k]
    total = sum(parts.values())
    achieved = total / (ms * 1e-3) / 1e12
    return dict(ms=ms, tokens=tokens, kept_per_layer=[int(np.sum(k)) for k in kpl], gen_s=gen_s,
                gflops={k: round(v / 1e9, 2) for k, v in parts.items()}, total_gflops=round(total / 1e9, 2),
                roof=dict(bound="mfma", achieved=round(achieved, 2), peak=MFMA_PEAK_TFLOPS["bf16"], unit="TFLOP/s",
                          frac=round(achieved / MFMA_PEAK_TFLOPS["bf16"], 4), traffic=None,
                          kernel="whole encoder step (model FLOPs as counted by model_flops)"))


def kernel_source_hash():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic():
    """HBM bytes per call of the two window-attention launches, from the committed counter
    measurement, if it was taken on the current kernel sources (else None)."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_call")


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


def roofline(flops, bytes_, kern_ms, pairs=None):
    """Roofline of the two window-attention launches against the largest of the MFMA, HBM and VALU floors
    (VALU: VALU_SLOTS_PER_PAIR issue slots per allowed pair and head, at VALU_PEAK_TOPS)."""
    t_mfma = flops / (MFMA_PEAK_TFLOPS["bf16"] * 1e12)
    t_hbm = bytes_ / (HBM_PEAK_GBS * 1e9)
    alu_ops = VALU_SLOTS_PER_PAIR * pairs if pairs is not None else 0.0
    t_alu = alu_ops / (VALU_PEAK_TOPS * 1e12)
    if t_alu >= max(t_mfma, t_hbm):
        achieved = alu_ops / (kern_ms * 1e-3) / 1e12
        roof = dict(bound="alu", achieved=round(achieved, 3), peak=round(VALU_PEAK_TOPS, 2),
                    unit="T VALU lane-op/s")
    elif t_mfma >= t_hbm:
        achieved = flops / (kern_ms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(achieved, 2), peak=MFMA_PEAK_TFLOPS["bf16"], unit="TFLOP/s")
    else:
        achieved = bytes_ / (kern_ms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s")
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["floor_mfma_us"] = round(t_mfma * 1e6, 2)
    roof["floor_hbm_us"] = round(t_hbm * 1e6, 2)
    roof["floor_alu_us"] = round(t_alu * 1e6, 2)
    roof["hbm_achieved_gbs"] = round(bytes_ / (kern_ms * 1e-3) / 1e9, 1)
    return roof


def measure(sc, si, torch, np, inp, theta, steps, warmup, dev="cuda:0", keep_ratio=None, causal=False):
    """Times `steps` steps (window attention with score partials, scores, prune + compaction of O) after
    `warmup` untimed ones.  theta None picks the median score of the valid non-global tokens (about half
    pruned), from one untimed step.  keep_ratio: prune by the top-k rule (sc_topk_prune_compact) instead of
    the threshold.  causal: the causal variant of the attention."""
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

    def step():
        sc.sc_window_attention(d, q, k, v, out=out, lse=lse, score_partials=sp, workspace=ws_attn)
        sc.sc_ltp_score(d, sp, scores=scores)
        if keep_ratio is None:
            sc.sc_ltp_prune_compact(d, scores, theta, True, [out], dsts=[oc], outs=outs, workspace=ws_prune)
        else:
            sc.sc_topk_prune_compact(d, scores, keep_ratio, True, [out], dsts=[oc], outs=outs, workspace=ws_prune)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    sc.sc_profile_window_kernel(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3 / steps
    ms = e0.elapsed_time(e1) / steps
    kern_ms, launches = sc.sc_profile_window_kernel_read()
    sc.sc_profile_window_kernel(False)
    kern_ms /= max(launches, 1)

    tokens = int(np.sum(inp["valid_len"]))
    pairs_w, pairs_g = algorithmic_counts(inp, causal)
    # algorithmic work of the two launches: Q.K^T and P.V once per allowed pair (the window rows and the
    # global rows); read Q, K, V, write O (bf16), the LSE and the score partials (fp32)
    flops = 4.0 * dd * H * (pairs_w + pairs_g)
    bytes_ = tokens * H * (4 * dd * 2 + 4) + sp.numel() * 4
    roof = roofline(flops, bytes_, kern_ms, pairs=H * (pairs_w + pairs_g))
    return dict(ms=ms, wall_ms=wall_ms, kern_ms=kern_ms, tokens=tokens, kept=outs["new_len"].cpu().tolist(),
                flops=flops, bytes=bytes_, roof=roof, theta=theta, pairs=H * (pairs_w + pairs_g))


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
        m = measure(sc, si, torch, np, inp, None, args.steps, args.warmup)
        print(json.dumps({
            "sweep": kind, "n": n, "window": w, "batch": B, "valid_tokens": m["tokens"],
            "allowed_pairs": m["pairs"], "ms_per_step": round(m["ms"], 4),
            "value": round(m["tokens"] / (m["ms"] * 1e-3), 1), "unit": "kept-token-layers/s",
            "attention_us": round(m["kern_ms"] * 1e3, 2), "ns_per_pair": round(m["kern_ms"] * 1e6 / m["pairs"], 4),
            "roofline": m["roof"], "kept_fraction": round(sum(m["kept"]) / m["tokens"], 3)}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the run, copy MIB MiB once on the GPU (a reference kernel of known traffic for "
                         "hardware counters)")
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="seq4096",
                    help="seq4096: B8 n4096 window 512, 32 global tokens (the headline line); lognormal: B64 n1024 "
                         "window 256, one global token, paper-shaped lognormal lengths; encoder: the 12-layer "
                         "stack; soft: training step (forward and backward) of one soft-pruned layer at seq4096")
    ap.add_argument("--prune", choices=("threshold", "topk"), default="threshold",
                    help="pruning rule of the step: the layer threshold (the paper's rule) or top-k by keep ratio")
    ap.add_argument("--keep-ratio", type=float, default=0.5, help="top-k rule: fraction of candidates kept")
    ap.add_argument("--causal", action="store_true",
                    help="the causal variant of the attention (keys after the query never attended); the "
                         "threshold is then the median score (the stored one belongs to the bidirectional scores)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the single measurement, sweep the window (n 4096) and the length (window "
                         "512), one JSON line per point")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the hot path runs on a single MI355X; --gpus {args.gpus} is not "
              "supported (sharding across GPUs is described, not built).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2310_07109_amd as sc
    import sc_inputs as si

    torch.cuda.set_device(0)
    dev = "cuda:0"
    if args.sweep:
        sweep(args, sc, si, torch, np)
        return
    cid, desc = WORKLOADS[args.workload]
    if cid == "soft":
        m = measure_soft(args, sc, si, torch, np, dev)
        line = {
            "metric": METRIC, "value": round(m["tokens"] / (m["ms"] * 1e-3), 1),
            "unit": "token-layers/s (training step)", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(m["ms"], 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": desc, "valid_tokens": m["tokens"], "threshold": m["theta"],
                       "temperature": m["temp"], "parallelism": "none (1 GPU)"},
            "roofline": m["roof"], "backward_ms": round(m["bwd_ms"], 4), "dtheta": m["dtheta"],
            "input_generation_s": round(m["gen_s"], 1)}
        if "cpu_baseline" in m:
            line["cpu_baseline"] = m["cpu_baseline"]
        print(json.dumps(line), flush=True)
        return
    if cid is None:
        m = measure_encoder(args, sc, si, torch, np, dev)
        print(json.dumps({
            "metric": METRIC, "value": round(m["tokens"] / (m["ms"] * 1e-3), 1), "unit": "kept-token-layers/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(m["ms"], 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": desc, "layer_input_tokens": m["tokens"], "kept_per_layer": m["kept_per_layer"],
                       "parallelism": "none (1 GPU)"},
            "model_gflops": m["gflops"], "model_gflops_total": m["total_gflops"], "roofline": m["roof"],
            "input_generation_s": round(m["gen_s"], 1)}), flush=True)
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
                causal=args.causal)
    theta = m["theta"]
    ms, tokens = m["ms"], m["tokens"]
    roof = m["roof"]
    # the recorded counters belong to the (bidirectional, threshold-pruned) seq4096 workload
    roof["traffic"] = recorded_traffic() if (args.workload == "seq4096" and not args.causal) else None
    roof["kernel"] = "k_attn_fwd<bf16> + k_attn_cols<bf16> (the two launches of the window attention)"
    roof["kernel_us"] = round(m["kern_ms"] * 1e3, 2)
    roof["algorithmic_flop"] = m["flops"]
    roof["algorithmic_bytes"] = m["bytes"]

    value = tokens / (ms * 1e-3)
    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "kept-token-layers/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": desc,
                   "batch": cfg.B, "seq_len": cfg.n, "heads": cfg.H, "head_dim": cfg.d, "window": cfg.window,
                   "global_tokens": cfg.n_global, "valid_tokens": tokens,
                   "pruning": (f"top-k, keep ratio {keep_ratio}" if keep_ratio is not None else
                               f"threshold {theta}"), "attention": "causal" if args.causal else "bidirectional",
                   "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "kept_per_sequence": m["kept"],
        "wall_ms_per_step": round(m["wall_ms"], 4),
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.default_threads()
        c0 = time.perf_counter()
        _, _, rs = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                           cfg.window, cfg.alpha, nthreads=threads, causal=args.causal)
        if keep_ratio is None:
            oracle.ltp_prune(rs.astype(np.float32), inp["valid_len"], inp["global_pos"], theta, 1)
        else:
            oracle.topk_prune(rs.astype(np.float32), inp["valid_len"], inp["global_pos"], keep_ratio, 1)
        cpu_s = time.perf_counter() - c0
        result["cpu_baseline"] = {"value": round(tokens / cpu_s, 1), "unit": "kept-token-layers/s", "cores": threads,
                                  "kind": "oracle",
                                  "sample": f"the whole workload once ({cfg.B} sequences, one layer: attention, "
                                            f"scores, pruning) in double precision, {cpu_s:.2f} s"}
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
