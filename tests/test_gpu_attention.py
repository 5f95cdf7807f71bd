"""GPU parity of sc_window_attention / sc_ltp_score / sc_ltp_prune_compact
against the CPU oracle, through the C ABI, on seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
import sc_inputs as si
from gpu_helpers import (NEAR_THETA, check_lse, check_out, check_scores, compare_keep, dev_i32, log, make_desc,
                         run_attention, stored_threshold, to_dev_storage)

pytestmark = pytest.mark.gpu

import paper_2310_07109_amd as sc  # noqa: E402


def small_case(name, dtype, B, n, H, window, G, len_range, mode="random", seed=7, lens=None, gp_override=None):
    cfg = si.AttnConfig(name, seed, B, n, H, 64, dtype, window, len_range, G, mode)
    inp = si.make_attention_inputs(cfg)
    if lens is not None:
        inp["valid_len"] = np.array(lens, np.int32)
        inp["global_pos"] = si.global_positions(seed, inp["valid_len"], G, mode)
    if gp_override is not None:
        inp["global_pos"] = np.array(gp_override, np.int32)
    return inp


SMALL = [
    # name, dtype, B, n, H, window, G, len range, extra
    ("single token", "bf16", 2, 1, 2, 4, 1, (1, 1), {}),
    ("ragged no global w0", "bf16", 2, 100, 3, 0, 0, (60, 100), {}),
    ("w1 equals w0", "f32", 1, 70, 2, 1, 0, (70, 70), {}),
    ("ragged varlen with empty seq", "bf16", 3, 200, 2, 16, 2, (0, 200), dict(lens=[0, 137, 200])),
    ("dense window", "bf16", 2, 300, 2, 1000, 1, (250, 300), {}),
    ("fp32 odd window G5", "f32", 2, 513, 2, 129, 5, (300, 513), {}),
    ("two slot chunks", "bf16", 1, 700, 2, 256, 70, (650, 700), {}),
    ("all tokens global", "bf16", 1, 96, 2, 8, 96, (96, 96), {}),
    ("global at last valid token", "bf16", 2, 160, 2, 32, 2, (160, 160),
     dict(gp_override=[[0, 159], [5, 159]])),
    ("unused slots", "f32", 2, 140, 2, 40, 4, (140, 140), dict(gp_override=[[3, 77, -1, -1], [-1, -1, -1, -1]])),
    ("600 global tokens", "bf16", 1, 1200, 2, 64, 600, (1100, 1200), {}),
    # the band-layout scores' one-key loads: n not a multiple of 4, and r = 259 not a multiple of 4, over many
    # 128-row blocks
    ("n 2050 window 512", "bf16", 1, 2050, 2, 512, 4, (1900, 2050), {}),
    ("r 259 fp32", "f32", 1, 2048, 2, 518, 3, (1800, 2048), {}),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_cases(case):
    name, dtype, B, n, H, window, G, lr, extra = case
    log(f"case {name}")
    inp = small_case(name, dtype, B, n, H, window, G, lr, **extra)
    ro, rl, rs = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                         window, inp["alpha"])
    g = run_attention(inp, band=True)
    check_out(g["out"], ro, dtype)
    check_lse(g["lse"], rl, inp["valid_len"])
    check_scores(g["scores"], rs, inp["valid_len"])
    check_scores(g["band_scores"], rs, inp["valid_len"])


def test_band_probs_layout_entries():
    """Paper layout: band entry (i, j) is P[i][i - r + j]; checked against the oracle's P via V = identity."""
    n, H, r = 64, 1, 5
    cfg = si.AttnConfig("band", 3, 1, n, H, 64, "f32", 2 * r, (n, n), 2, "random")
    inp = si.make_attention_inputs(cfg)
    gp = inp["global_pos"]
    # oracle probabilities: V = identity rows gives O[i] = P[i, :64]
    eye = np.zeros((1, n, H, 64))
    eye[0, :, 0, :] = np.eye(n, 64)
    P, _, _ = oracle.sparse_attention(inp["q64"], inp["k64"], eye, inp["valid_len"], gp, 2 * r, inp["alpha"])
    P = P[0, :, 0, :]
    g = run_attention(inp, band=True)
    bp = g["band_probs"].cpu().numpy()
    bw = 2 * r + 1
    band = bp[: n * bw].reshape(n, bw)
    G = gp.shape[1]
    gcol = bp[n * bw: n * bw + n * G].reshape(n, G)
    grow = bp[n * bw + n * G:].reshape(G, n)
    glob = set(gp[0].tolist())
    for i in range(n):
        for j in range(bw):
            k = i - r + j
            want = P[i, k] if (0 <= k < n and i not in glob and k not in glob) else 0.0
            assert abs(band[i, j] - want) <= 1e-5 * abs(want) + 1e-9
        for s, p in enumerate(gp[0]):
            want = P[i, p] if i not in glob else 0.0
            assert abs(gcol[i, s] - want) <= 1e-5 * abs(want) + 1e-9
    for s, p in enumerate(gp[0]):
        np.testing.assert_allclose(grow[s], P[p], rtol=1e-5, atol=1e-9)


_CACHE = {}


def config_run(cid):
    if cid not in _CACHE:
        cfg = si.CONFIGS[cid]
        log(f"config {cid}: generating inputs")
        inp = si.make_attention_inputs(cfg)
        log(f"config {cid}: oracle")
        ref = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                      inp["window"], inp["alpha"])
        log(f"config {cid}: gpu")
        g = run_attention(inp, band=True)
        _CACHE[cid] = (inp, ref, g)
    return _CACHE[cid]


@pytest.mark.parametrize("cid", [1, 2, 4, 6])
def test_config_attention_and_scores(cid):
    inp, (ro, rl, rs), g = config_run(cid)
    err = check_out(g["out"], ro, inp["dtype"])
    check_lse(g["lse"], rl, inp["valid_len"])
    worst = check_scores(g["scores"], rs, inp["valid_len"])
    # the paper's path: every probability stored in the band layout, scores summed from it
    worst_band = check_scores(g["band_scores"], rs, inp["valid_len"])
    log(f"config {cid}: max |dO| {err:.3g}, worst score rel err {worst:.3g} (band layout {worst_band:.3g})")


@pytest.mark.parametrize("cid", [1, 2, 4, 6])
def test_config_prune_compact(cid):
    inp, (ro, rl, rs), g = config_run(cid)
    cfg = si.CONFIGS[cid]
    theta = cfg.thresholds[0] if cfg.thresholds[0] is not None else stored_threshold(cid)
    d = g["desc"]
    # 1) the whole path: GPU scores -> GPU keep
    keep, nl, ngp, orig, (oc,) = sc.sc_ltp_prune_compact(d, g["scores_t"], theta, True, [g["out_t"]])
    keep, nl = keep.cpu().numpy(), nl.cpu().numpy()
    excl, dis = compare_keep(keep, nl, rs, theta, inp["valid_len"], inp["global_pos"], tag=f"config {cid} keep")
    log(f"config {cid}: kept {nl.tolist()} of {inp['valid_len'].tolist()}")
    # 2) compaction on the oracle's float32 scores is bit-exact
    s32 = torch.from_numpy(rs.astype(np.float32)).cuda()
    keep2, nl2, ngp2, orig2, (oc2,) = sc.sc_ltp_prune_compact(d, s32, theta, True, [g["out_t"]])
    rk, rnl, rngp, rorig = oracle.ltp_prune(rs.astype(np.float32), inp["valid_len"], inp["global_pos"], theta, 1)
    assert np.array_equal(keep2.cpu().numpy(), rk) and np.array_equal(nl2.cpu().numpy(), rnl)
    assert np.array_equal(ngp2.cpu().numpy(), rngp) and np.array_equal(orig2.cpu().numpy(), rorig)
    src = g["out_t"].view(torch.int16).cpu().numpy() if inp["dtype"] == "bf16" else g["out_t"].cpu().numpy()
    dst = oc2.view(torch.int16).cpu().numpy() if inp["dtype"] == "bf16" else oc2.cpu().numpy()
    for b in range(d.B):
        assert np.array_equal(dst[b, :rnl[b]], src[b, rk[b, :rnl[b]]])


@pytest.mark.parametrize("cid", [5, "5b"])
def test_config5_three_passes(cid):
    """Three successive prune passes on the compacted Q, K, V (renumbered positions, remapped globals); the
    literal workload (rank-4 spike on K) and variant 5b (the spike on Q as well, heavy-tailed scores)."""
    cfg = si.CONFIGS[cid]
    log(f"config {cid}: generating inputs")
    inp = si.make_attention_inputs(cfg)
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    q64, k64, v64 = inp["q64"], inp["k64"], inp["v64"]
    vl, gp = inp["valid_len"].copy(), inp["global_pos"].copy()
    for p, theta in enumerate(cfg.thresholds):
        log(f"config {cid} pass {p}: L={vl.tolist()}")
        ro, rl, rs = oracle.sparse_attention(q64, k64, v64, vl, gp, cfg.window, cfg.alpha)
        d = sc.Desc(cfg.B, cfg.n, cfg.H, cfg.window, dev_i32(vl), dev_i32(gp), cfg.alpha, sc.SC_BF16)
        out, lse, sp, _ = sc.sc_window_attention(d, q, k, v)
        scores = sc.sc_ltp_score(d, sp)
        check_out(out.float().cpu().numpy(), ro, "bf16")
        check_scores(scores.cpu().numpy(), rs, vl)
        keep, nl, ngp, _, (q2, k2, v2) = sc.sc_ltp_prune_compact(d, scores, theta, True, [q, k, v])
        keep_np, nl_np = keep.cpu().numpy(), nl.cpu().numpy()
        excl, dis = compare_keep(keep_np, nl_np, rs, theta, vl, gp, tag=f"config {cid} pass {p} keep")
        log(f"config {cid} pass {p}: kept {nl_np.tolist()}")
        # continue the oracle on the GPU's kept lists (identical outside the near-theta band)
        rk = keep_np
        q64c, k64c, v64c = (np.zeros_like(x) for x in (q64, k64, v64))
        for b in range(cfg.B):
            idx = rk[b, :nl_np[b]]
            q64c[b, :len(idx)], k64c[b, :len(idx)], v64c[b, :len(idx)] = q64[b, idx], k64[b, idx], v64[b, idx]
        q64, k64, v64 = q64c, k64c, v64c
        vl = nl_np.astype(np.int32)
        gp = ngp.cpu().numpy()
        q, k, v = q2, k2, v2


def test_determinism():
    inp = small_case("det", "bf16", 2, 777, 4, 200, 9, (500, 777))
    a = run_attention(inp)
    b = run_attention(inp)
    for key in ("out", "lse", "scores"):
        assert np.array_equal(a[key], b[key]), key


def test_prune_edge_cases():
    inp = small_case("edges", "bf16", 3, 300, 2, 64, 3, (0, 300), lens=[0, 1, 300])
    g = run_attention(inp)
    d = g["desc"]
    ro, rl, rs = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                         64, inp["alpha"])
    for theta, kg in ((-1.0, 1), (1.0, 1), (1.0, 0), (0.0, 0), (float(np.float32(rs[2, 10])), 1)):
        s32 = torch.from_numpy(rs.astype(np.float32)).cuda()
        keep, nl, ngp, orig, _ = sc.sc_ltp_prune_compact(d, s32, theta, kg)
        rk, rnl, rngp, rorig = oracle.ltp_prune(rs.astype(np.float32), inp["valid_len"], inp["global_pos"], theta,
                                                kg)
        assert np.array_equal(keep.cpu().numpy(), rk) and np.array_equal(nl.cpu().numpy(), rnl)
        assert np.array_equal(ngp.cpu().numpy(), rngp) and np.array_equal(orig.cpu().numpy(), rorig)


def test_orig_index_composition_and_poisoned_tail():
    """orig_idx_in composes; destination rows beyond new_len are left untouched."""
    inp = small_case("orig", "bf16", 2, 256, 2, 32, 1, (200, 256), mode="first")
    g = run_attention(inp)
    d = g["desc"]
    oin = torch.randint(0, 10000, (2, 256), dtype=torch.int32, device="cuda")
    dst = torch.full_like(g["out_t"], float("nan"))
    keep, nl, _, orig, (oc,) = sc.sc_ltp_prune_compact(d, g["scores_t"], 0.004, True, [g["out_t"]], dsts=[dst],
                                                       orig_idx_in=oin)
    keep, nl, orig, oin = keep.cpu().numpy(), nl.cpu().numpy(), orig.cpu().numpy(), oin.cpu().numpy()
    oc = oc.float().cpu().numpy()
    for b in range(2):
        m = nl[b]
        assert np.array_equal(orig[b, :m], oin[b, keep[b, :m]]) and np.all(orig[b, m:] == -1)
        assert np.all(np.isnan(oc[b, m:])) and not np.isnan(oc[b, :m]).any()


def _topk_compare(d, scores_np, vl, gp, ratio, keep_global, rows=None):
    """GPU top-k compaction of float32 scores against the oracle, bit-exact (indices and gathered rows)."""
    s32 = torch.from_numpy(np.ascontiguousarray(scores_np, dtype=np.float32)).to("cuda:0")
    tensors = [rows] if rows is not None else []
    keep, nl, ngp, orig, dsts = sc.sc_topk_prune_compact(d, s32, ratio, keep_global, tensors)
    rk, rnl, rngp, rorig = oracle.topk_prune(scores_np, vl, gp, ratio, keep_global)
    assert np.array_equal(nl.cpu().numpy(), rnl), (ratio, keep_global)
    assert np.array_equal(keep.cpu().numpy(), rk)
    assert np.array_equal(orig.cpu().numpy(), rorig)
    if ngp is not None:
        assert np.array_equal(ngp.cpu().numpy(), rngp)
    if rows is not None:
        src, dst = rows.view(torch.int16).cpu().numpy(), dsts[0].view(torch.int16).cpu().numpy()
        for b in range(len(rnl)):
            assert np.array_equal(dst[b, :rnl[b]], src[b, rk[b, :rnl[b]]])
    return rnl


@pytest.mark.parametrize("cid", [2, 4, 6])
def test_config_topk_prune(cid):
    """Top-k rule on the oracle's float32 scores of a workload: bit-exact keep lists and compaction."""
    inp, (ro, rl, rs), g = config_run(cid)
    d = g["desc"]
    for ratio in (0.0, 0.3, 0.5, 0.9, 1.0):
        for kg in (1, 0):
            nl = _topk_compare(d, rs.astype(np.float32), inp["valid_len"], inp["global_pos"], ratio, kg,
                               rows=g["out_t"] if (ratio == 0.5 and kg) else None)
    log(f"config {cid}: top-k ratio 1.0 keeps {nl.tolist()}")


@pytest.mark.parametrize("n", [2600, 9000], ids=["registers", "chunked"])
def test_topk_ties_signs_and_lengths(n):
    """Ties everywhere (scores on 3 levels), negative scores and both zeros, lengths 0 / 1 / n / ragged over
    several 1024-token chunks; n = 2600 takes the path that holds a thread's tokens in registers (up to 8192
    tokens), n = 9000 the chunked one."""
    rng = np.random.default_rng(5)
    B, G = 6, 5
    vl = np.array([0, 1, n, 1500, 2047, 999], np.int32)
    gp = np.full((B, G), -1, np.int32)
    for b in range(B):
        if vl[b]:
            gp[b, :min(G, vl[b])] = np.sort(rng.choice(vl[b], size=min(G, vl[b]), replace=False))
    levels = np.array([-0.5, -0.0, 0.0, 0.25, 0.25, 1.0], np.float32)
    s = levels[rng.integers(0, len(levels), (B, n))]
    d = sc.Desc(B, n, 2, 8, dev_i32(vl), dev_i32(gp), 0.125, sc.SC_BF16)
    rows = torch.from_numpy(rng.integers(-30000, 30000, (B, n, 16)).astype(np.int16)).to("cuda:0").view(torch.bfloat16)
    for ratio in (0.0, 1e-4, 0.2, 1.0 / 3.0, 0.5, 0.75, 1.0):
        for kg in (1, 0):
            _topk_compare(d, s, vl, gp, ratio, kg, rows=rows if kg else None)


CAUSAL = [
    # name, B, n, H, window, G, len range, extra (bf16)
    ("causal single token", 2, 1, 2, 4, 1, (1, 1), {}),
    ("causal ragged no global", 2, 300, 3, 64, 0, (200, 300), {}),
    ("causal w0", 1, 70, 2, 0, 0, (70, 70), {}),
    ("causal ragged with empty seq", 3, 260, 2, 40, 2, (0, 260), dict(lens=[0, 137, 260])),
    ("causal dense window", 2, 300, 2, 1000, 1, (250, 300), {}),
    ("causal two slot chunks", 1, 700, 2, 256, 70, (650, 700), {}),
    ("causal all tokens global", 1, 96, 2, 8, 96, (96, 96), {}),
    ("causal global at last valid token", 2, 160, 2, 32, 2, (160, 160), dict(gp_override=[[0, 159], [5, 159]])),
    ("causal 600 global tokens", 1, 1200, 2, 64, 600, (1100, 1200), {}),
    ("causal long window ragged", 2, 2000, 2, 700, 5, (1500, 2000), {}),
]


@pytest.mark.parametrize("case", CAUSAL, ids=[c[0] for c in CAUSAL])
def test_causal_small_cases(case):
    """Causal variant: keys after the query are never attended (band and global strips alike)."""
    name, B, n, H, window, G, lr, extra = case
    log(f"case {name}")
    inp = small_case(name, "bf16", B, n, H, window, G, lr, **extra)
    ro, rl, rs = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                         window, inp["alpha"], causal=True)
    d = make_desc(inp)
    d.causal = 1
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    out, lse, sp, _ = sc.sc_window_attention(d, q, k, v, lse=True, score_partials=True)
    scores = sc.sc_ltp_score(d, sp)
    torch.cuda.synchronize()
    check_out(out.float().cpu().numpy(), ro, "bf16")
    check_lse(lse.cpu().numpy(), rl, inp["valid_len"])
    check_scores(scores.cpu().numpy(), rs, inp["valid_len"])


def test_causal_config4_attention_scores_and_pruning():
    """Causal variant of the seq-4096 workload at full size: O, LSE, scores, and the compaction on the oracle's
    scores (bit-exact) and on the GPU's own scores (kept lists, near-threshold tokens excluded)."""
    cfg = si.CONFIGS[4]
    inp = si.make_attention_inputs(cfg)
    log("causal config 4: oracle")
    ro, rl, rs = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                         inp["window"], inp["alpha"], causal=True)
    d = make_desc(inp)
    d.causal = 1
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    out, lse, sp, _ = sc.sc_window_attention(d, q, k, v, lse=True, score_partials=True)
    scores = sc.sc_ltp_score(d, sp)
    torch.cuda.synchronize()
    err = check_out(out.float().cpu().numpy(), ro, "bf16")
    check_lse(lse.cpu().numpy(), rl, inp["valid_len"])
    worst = check_scores(scores.cpu().numpy(), rs, inp["valid_len"])
    theta = float(np.median(rs[0, :int(inp["valid_len"][0])]))
    keep, nl, ngp, orig, _ = sc.sc_ltp_prune_compact(d, scores, theta, True)
    compare_keep(keep.cpu().numpy(), nl.cpu().numpy(), rs, theta, inp["valid_len"], inp["global_pos"],
                 tag="causal config 4 keep")
    log(f"causal config 4: max |dO| {err:.3g}, worst score rel err {worst:.3g}, kept {nl.cpu().tolist()}")


@pytest.mark.parametrize("kg", [1, 0])
def test_prune_compact_fused_and_fallback_paths(kg):
    """The one-launch threshold prune (16-byte aligned rows, up to four tensors) and the two-kernel path it
    falls back to (any row that is not 16-byte aligned) give identical survivor lists, lengths, renumbered
    globals and composed indices, equal to the oracle's, and copy the same rows.  Ragged lengths (an empty
    sequence), n not a multiple of the 64-token chunk, unused global slots, ties at the threshold."""
    B, n, G = 3, 1000, 40
    vl = np.array([0, 537, 1000], np.int32)
    gp = si.global_positions(11, vl, G, "random")
    gp[2, -5:] = -1  # unused slots at the end of one row
    u = si.uniform(11, 5, B * n).reshape(B, n)
    scores = (u * 2e-3).astype(np.float32)
    theta = float(np.float32(scores[2, 123]))  # a score equal to the threshold is pruned
    d = sc.Desc(B, n, 2, 64, dev_i32(vl), dev_i32(gp), 0.125, sc.SC_BF16)
    s_dev = torch.from_numpy(scores).cuda()
    oin = torch.from_numpy(si.randint(11, 6, B * n, 0, 1 << 20).reshape(B, n).astype(np.int32)).cuda()
    # four aligned tensors (rows of 16, 48, 256 and 1536 bytes) take the one-launch path
    aligned = [torch.from_numpy(si.randint(11, 7 + i, B * n * w, -30000, 30000).reshape(B, n, w).astype(np.int16)).cuda()
               for i, w in enumerate((8, 24, 128, 768))]
    ka, nla, gpa, oa, da = sc.sc_ltp_prune_compact(d, s_dev, theta, kg, aligned, orig_idx_in=oin)
    # one 6-byte row makes the call take the scan + gather kernels
    odd = torch.from_numpy(si.randint(11, 12, B * n * 3, -30000, 30000).reshape(B, n, 3).astype(np.int16)).cuda()
    kb, nlb, gpb, ob, db = sc.sc_ltp_prune_compact(d, s_dev, theta, kg, [aligned[0], odd], orig_idx_in=oin)
    rk, rnl, rngp, rorig = oracle.ltp_prune(scores, vl, gp, theta, kg, orig_in=oin.cpu().numpy())
    assert 0 < rnl[1] < vl[1] and 0 < rnl[2] < vl[2] and rnl[0] == 0
    for k_, nl_, gp_, o_ in ((ka, nla, gpa, oa), (kb, nlb, gpb, ob)):
        assert np.array_equal(k_.cpu().numpy(), rk) and np.array_equal(nl_.cpu().numpy(), rnl)
        assert np.array_equal(gp_.cpu().numpy(), rngp)
        assert np.array_equal(o_.cpu().numpy(), rorig)
    for src, dst in list(zip(aligned, da)) + [(odd, db[1]), (aligned[0], db[0])]:
        s_np, d_np = src.cpu().numpy(), dst.cpu().numpy()
        for b in range(B):
            assert np.array_equal(d_np[b, :rnl[b]], s_np[b, rk[b, :rnl[b]]])
    log(f"fused / fallback prune (keep_global={kg}): kept {rnl.tolist()}, globals kept "
        f"{[(int((rngp[b] >= 0).sum())) for b in range(B)]}")


# Batches of sequences longer than 4096 tokens take the pair-by-pair dispatch of the attention blocks (shorter ones
# the span order, which every case above runs); these cases run the pair order against the oracle.
PAIR_ORDER = [
    # name, dtype, B, n, H, window, G, len range, causal
    ("pair order bf16 two slot chunks", "bf16", 2, 4224, 2, 256, 40, (3000, 4224), False),
    ("pair order fp32", "f32", 1, 4160, 2, 128, 3, (4100, 4160), False),
    ("pair order causal", "bf16", 2, 4160, 2, 512, 33, (2500, 4160), True),
]


@pytest.mark.parametrize("case", PAIR_ORDER, ids=[c[0] for c in PAIR_ORDER])
def test_pair_order_cases(case):
    name, dtype, B, n, H, window, G, lr, causal = case
    log(f"case {name}")
    inp = small_case(name, dtype, B, n, H, window, G, lr)
    ro, rl, rs = oracle.sparse_attention(inp["q64"], inp["k64"], inp["v64"], inp["valid_len"], inp["global_pos"],
                                         window, inp["alpha"], causal=causal)
    d = make_desc(inp)
    d.causal = int(causal)
    q, k, v = (to_dev_storage(inp[x], dtype) for x in ("q", "k", "v"))
    out, lse, sp, _ = sc.sc_window_attention(d, q, k, v, lse=True, score_partials=True)
    scores = sc.sc_ltp_score(d, sp)
    torch.cuda.synchronize()
    check_out(out.float().cpu().numpy(), ro, dtype)
    check_lse(lse.cpu().numpy(), rl, inp["valid_len"])
    check_scores(scores.cpu().numpy(), rs, inp["valid_len"])


@pytest.mark.parametrize("causal", [0, 1])
def test_dispatch_order_invariance(causal):
    """The same sequences in an n = 4096 batch (span order) and, padded, in an n = 4160 batch (pair order) give
    bit-identical outputs, LSE and scores on their valid rows: every block computes the same values, in the same
    order, whichever order the blocks are dispatched in."""
    inp = small_case("order", "bf16", 3, 4096, 2, 512, 32, (1000, 4096), lens=[4096, 2345, 1000])
    n2 = 4160
    res = []
    for n in (4096, n2):
        q, k, v = (np.zeros((inp["B"], n) + inp[x].shape[2:], inp[x].dtype) for x in ("q", "k", "v"))
        q[:, :4096], k[:, :4096], v[:, :4096] = inp["q"], inp["k"], inp["v"]
        d = sc.Desc(inp["B"], n, inp["H"], inp["window"], dev_i32(inp["valid_len"]), dev_i32(inp["global_pos"]),
                    inp["alpha"], sc.SC_BF16)
        d.causal = causal
        out, lse, sp, _ = sc.sc_window_attention(d, *(to_dev_storage(x, "bf16") for x in (q, k, v)), lse=True,
                                                 score_partials=True)
        scores = sc.sc_ltp_score(d, sp)
        torch.cuda.synchronize()
        res.append((out.view(torch.int16).cpu().numpy(), lse.cpu().numpy(), scores.cpu().numpy()))
    for b, L in enumerate(inp["valid_len"]):
        assert np.array_equal(res[0][0][b, :L], res[1][0][b, :L]), f"output of sequence {b} differs"
        assert np.array_equal(res[0][1][b, :, :L], res[1][1][b, :, :L]), f"lse of sequence {b} differs"
        assert np.array_equal(res[0][2][b, :L], res[1][2][b, :L]), f"scores of sequence {b} differ"
    log(f"dispatch orders bit-identical (causal {causal})")
