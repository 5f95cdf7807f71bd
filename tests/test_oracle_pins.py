"""Pins of the CPU oracle against things other than itself (no GPU).

Each check pins one or more parts of the oracle against brute force on tiny
inputs, a library routine the method reduces to, a closed form, an invariant
or a value the paper prints.  ``test_oracle_mutants.py`` re-runs these checks
on deliberately broken copies of the oracle to show that each plausible
mistake is caught by at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import sc_inputs as si

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------- helpers --
def rand_case(seed, B=2, n=24, H=3, d=8, window=None, G=None, full=False, scale=0.7):
    rng = np.random.default_rng(seed)
    window = int(rng.integers(0, n)) if window is None else window
    q = rng.standard_normal((B, n, H, d)) * scale
    k = rng.standard_normal((B, n, H, d)) * scale
    v = rng.standard_normal((B, n, H, d))
    vl = np.full(B, n, np.int32) if full else rng.integers(1, n + 1, B).astype(np.int32)
    G = int(rng.integers(0, 4)) if G is None else G
    gp = np.full((B, max(G, 1)), -1, np.int32)
    for b in range(B):
        g = rng.choice(vl[b], size=min(G, vl[b]), replace=False) if G else []
        gp[b, :len(g)] = np.sort(g)
    return q, k, v, vl, gp, window


def allowed_matrix(n, L, r, gflags, causal=False):
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    m = (np.abs(i - j) <= r) | gflags[:, None] | gflags[None, :]
    if causal:
        m = m & (j <= i)
    return m & (i < L) & (j < L)


def brute_force(q, k, v, vl, gp, window, alpha, causal=False):
    """Explicit n x n masked softmax attention in numpy (tiny inputs only)."""
    B, n, H, d = q.shape
    r = window // 2
    out = np.zeros_like(q)
    lse = np.full((B, H, n), -np.inf)
    colsum = np.zeros((B, H, n))
    for b in range(B):
        L = int(vl[b])
        gf = np.zeros(n, bool)
        for p in gp[b]:
            if 0 <= p < L:
                gf[p] = True
        M = allowed_matrix(n, L, r, gf, causal)
        for h in range(H):
            S = alpha * q[b, :, h, :] @ k[b, :, h, :].T
            S = np.where(M, S, -np.inf)
            for i in range(L):
                m = S[i].max()
                e = np.where(M[i], np.exp(S[i] - m), 0.0)
                z = e.sum()
                p = e / z
                out[b, i, h] = p @ v[b, :, h, :]
                lse[b, h, i] = m + math.log(z)
                colsum[b, h] += p
    scores = np.zeros((B, n))
    for b in range(B):
        L = int(vl[b])
        if L:
            scores[b, :L] = colsum[b, :, :L].sum(0) / (H * L)
    return out, lse, scores


def run(q, k, v, vl, gp, window, alpha=0.35, **kw):
    return oracle.sparse_attention(q, k, v, vl, gp, window, alpha, **kw)


# ------------------------------------------------------------------ checks --
def check_brute_force():
    for seed in range(12):
        q, k, v, vl, gp, w = rand_case(seed)
        o, l, s = run(q, k, v, vl, gp, w)
        bo, bl, bs = brute_force(q, k, v, vl, gp, w, 0.35)
        np.testing.assert_allclose(o, bo, rtol=0, atol=1e-12)
        fin = np.isfinite(bl)
        assert np.array_equal(fin, np.isfinite(l))
        np.testing.assert_allclose(l[fin], bl[fin], rtol=0, atol=1e-12)
        np.testing.assert_allclose(s, bs, rtol=0, atol=1e-13)


def check_causal_brute_force():
    """Causal variant (keys after the query never attended, band and global strips alike) against the explicit
    n x n mask."""
    for seed in range(12):
        q, k, v, vl, gp, w = rand_case(300 + seed)
        o, l, s = run(q, k, v, vl, gp, w, causal=True)
        bo, bl, bs = brute_force(q, k, v, vl, gp, w, 0.35, causal=True)
        np.testing.assert_allclose(o, bo, rtol=0, atol=1e-12)
        fin = np.isfinite(bl)
        assert np.array_equal(fin, np.isfinite(l))
        np.testing.assert_allclose(l[fin], bl[fin], rtol=0, atol=1e-12)
        np.testing.assert_allclose(s, bs, rtol=0, atol=1e-13)


def check_causal_dense_is_library_causal_attention():
    """A window covering the sequence, no global token, causal: torch's causal SDPA (float64); the first token
    attends only to itself; the scores still sum to one."""
    q, k, v, vl, gp, _ = rand_case(310, n=20, full=True, G=0)
    o, l, s = run(q, k, v, vl, gp, 1000, causal=True)
    Q, K, V = (torch.from_numpy(x).permute(0, 2, 1, 3) for x in (q, k, v))
    O = torch.nn.functional.scaled_dot_product_attention(Q, K, V, scale=0.35, is_causal=True)
    np.testing.assert_allclose(o, O.permute(0, 2, 1, 3).numpy(), atol=1e-12)
    assert np.array_equal(o[:, 0], v[:, 0])
    np.testing.assert_allclose(l[:, :, 0], 0.35 * np.einsum("bhd,bhd->bh", q[:, 0], k[:, 0]), atol=1e-12)
    np.testing.assert_allclose(s.sum(1), 1.0, atol=1e-12)


def _sdpa(q, k, v, alpha):
    """Dense attention by torch's library routine, float64; [B, n, H, d] layout."""
    Q, K, V = (torch.from_numpy(x).permute(0, 2, 1, 3) for x in (q, k, v))
    O = torch.nn.functional.scaled_dot_product_attention(Q, K, V, scale=alpha)
    S = alpha * Q @ K.transpose(-1, -2)
    lse = torch.logsumexp(S, -1)
    P = torch.softmax(S, -1)
    n = q.shape[1]
    scores = P.sum(2).mean(1) / n  # sum over queries, mean over heads, / L
    return O.permute(0, 2, 1, 3).numpy(), lse.numpy(), scores.numpy()


def check_window_covers_sequence_is_dense():
    q, k, v, vl, gp, _ = rand_case(100, n=20, full=True, G=0)
    for w in (40, 41, 1000):
        o, l, s = run(q, k, v, vl, gp, w)
        ro, rl, rs = _sdpa(q, k, v, 0.35)
        np.testing.assert_allclose(o, ro, atol=1e-12)
        np.testing.assert_allclose(l, rl, atol=1e-12)
        np.testing.assert_allclose(s, rs, atol=1e-14)


def check_all_global_is_dense():
    q, k, v, vl, _, _ = rand_case(101, n=16, full=True)
    gp = np.tile(np.arange(16, dtype=np.int32), (q.shape[0], 1))
    o, l, s = run(q, k, v, vl, gp, 2)
    ro, rl, rs = _sdpa(q, k, v, 0.35)
    np.testing.assert_allclose(o, ro, atol=1e-12)
    np.testing.assert_allclose(s, rs, atol=1e-14)


def check_zero_window_no_global():
    """r = 0 and no global token: every query attends only to itself."""
    q, k, v, vl, gp, _ = rand_case(102, G=0)
    gp[:] = -1
    for w in (0, 1):
        o, l, s = run(q, k, v, vl, gp, w)
        B, n = q.shape[:2]
        for b in range(B):
            L = int(vl[b])
            assert np.array_equal(o[b, :L], v[b, :L])           # P = 1 exactly
            assert np.all(o[b, L:] == 0)
            assert np.all(s[b, :L] == 1.0 / L) and np.all(s[b, L:] == 0)
            self_logit = 0.35 * np.einsum("nhd,nhd->hn", q[b, :L], k[b, :L])
            np.testing.assert_allclose(l[b, :, :L], self_logit, rtol=1e-14, atol=1e-15)
            assert np.all(np.isneginf(l[b, :, L:]))


def check_constant_values():
    q, k, v, vl, gp, w = rand_case(103)
    c = np.linspace(-1, 1, q.shape[-1])
    v[:] = c
    o, _, _ = run(q, k, v, vl, gp, w)
    for b in range(q.shape[0]):
        np.testing.assert_allclose(o[b, :vl[b]], np.broadcast_to(c, o[b, :vl[b]].shape), atol=1e-14)


def check_zero_queries_rational_scores():
    """Q = 0 makes every row uniform over its neighbour set: exact rational scores by counting."""
    for seed in (104, 105, 106):
        q, k, v, vl, gp, w = rand_case(seed, n=20)
        q[:] = 0.0
        _, _, s = run(q, k, v, vl, gp, w)
        r = w // 2
        for b in range(q.shape[0]):
            L = int(vl[b])
            g = set(int(p) for p in gp[b] if 0 <= p < L)
            nb = [[j for j in range(L) if abs(i - j) <= r or i in g or j in g] for i in range(L)]
            for kk in range(L):
                exact = sum((Fraction(1, len(nb[i])) for i in range(L) if kk in nb[i]), Fraction(0)) / L
                assert abs(s[b, kk] - float(exact)) < 1e-15


def check_score_invariants():
    for seed in range(200, 206):
        q, k, v, vl, gp, w = rand_case(seed, n=40)
        o, l, s, cs = run(q, k, v, vl, gp, w, want_colsum=True)
        for b in range(q.shape[0]):
            L = int(vl[b])
            np.testing.assert_allclose(s[b].sum(), 1.0, atol=1e-13)          # sum over tokens is one
            np.testing.assert_allclose(cs[b].sum(-1), np.full(q.shape[2], L), atol=1e-11)  # rows sum to 1
            assert np.all(s[b, L:] == 0) and np.all(s[b, :L] > 0)


def check_reflection_symmetry():
    q, k, v, vl, gp, w = rand_case(300, n=30, full=True, G=2)
    o, l, s = run(q, k, v, vl, gp, w)
    n = q.shape[1]
    gpr = np.where(gp >= 0, n - 1 - gp, -1)
    gpr = np.sort(np.where(gpr < 0, 10 ** 6, gpr), 1)
    gpr = np.where(gpr == 10 ** 6, -1, gpr).astype(np.int32)
    o2, l2, s2 = run(q[:, ::-1], k[:, ::-1], v[:, ::-1], vl, gpr, w)
    np.testing.assert_allclose(o2[:, ::-1], o, atol=1e-13)
    np.testing.assert_allclose(s2[:, ::-1], s, atol=1e-14)


def check_head_permutation():
    q, k, v, vl, gp, w = rand_case(301, H=4)
    perm = [2, 0, 3, 1]
    o, l, s = run(q, k, v, vl, gp, w)
    o2, l2, s2 = run(q[:, :, perm], k[:, :, perm], v[:, :, perm], vl, gp, w)
    np.testing.assert_allclose(o2, o[:, :, perm], atol=0)
    np.testing.assert_allclose(s2, s, atol=1e-15)


def check_sec55_example_structure():
    """Paper's worked example (Sec. 5.5): ten tokens, specials 1st and 8th, window 3.

    With Q = 0 the softmax is uniform over the allowed keys and V = identity
    makes the output row i equal P[i, :], so the oracle's support is read off.
    """
    lines = [ln for ln in open(os.path.join(GOLDEN, "sec55_example_mask.txt")) if not ln.startswith("#")]
    glob = [int(x) for x in lines[0].split()[1:]]
    window = int(lines[1].split()[1])
    M = np.array([[c == "1" for c in ln.strip()] for ln in lines[2:12]])
    n = 10
    q = np.zeros((1, n, 1, n))
    k = np.random.default_rng(0).standard_normal((1, n, 1, n))
    v = np.eye(n).reshape(1, n, 1, n)
    o, _, _ = run(q, k, v, np.array([n], np.int32), np.array([glob], np.int32), window)
    P = o[0, :, 0, :]
    assert np.array_equal(P > 0, M)
    np.testing.assert_allclose(P.sum(1), 1.0, atol=1e-15)
    np.testing.assert_allclose(P[M], np.repeat(1.0 / M.sum(1), M.sum(1)), atol=1e-15)


def check_padding_is_invisible():
    """Padding tokens neither attend nor are attended: changing them changes nothing."""
    q, k, v, vl, gp, w = rand_case(302, n=32)
    vl[:] = [20, 9]
    o, l, s = run(q, k, v, vl, gp, w)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for b, L in enumerate(vl):
        q2[b, L:] = 7.0
        k2[b, L:] = -3.0
        v2[b, L:] = 11.0
    o2, l2, s2 = run(q2, k2, v2, vl, gp, w)
    assert np.array_equal(o, o2) and np.array_equal(s, s2)
    # and a shorter padded copy gives the same valid outputs
    o3, _, s3 = run(q[:1, :20], k[:1, :20], v[:1, :20], vl[:1], gp[:1], w)
    np.testing.assert_allclose(o3[0], o[0, :20], atol=0)
    np.testing.assert_allclose(s3[0], s[0, :20], atol=0)


def brute_prune(s32, vl, gp, theta, keep_global, orig_in=None):
    B, n = s32.shape
    out = []
    for b in range(B):
        L = int(vl[b])
        g = [int(p) for p in gp[b] if 0 <= p < L]
        kept = [kk for kk in range(L) if s32[b, kk] > np.float32(theta) or (keep_global and kk in g)]
        ng = [kept.index(p) for p in g if p in kept]
        orig = [(orig_in[b, kk] if orig_in is not None else kk) for kk in kept]
        out.append((kept, ng, orig))
    return out


def check_prune_brute_force():
    rng = np.random.default_rng(7)
    for trial in range(20):
        B, n, G = 3, 50, 4
        s = rng.random((B, n)).astype(np.float32) * 0.05
        vl = rng.integers(0, n + 1, B).astype(np.int32)
        gp = np.full((B, G), -1, np.int32)
        for b in range(B):
            g = rng.choice(max(vl[b], 1), size=min(G, vl[b]), replace=False) if vl[b] else []
            gp[b, :len(g)] = np.sort(g)
        theta = float(rng.choice([-1.0, 0.0, 0.01, 0.025, 0.049, float(s[0, 3])]))
        kg = int(trial % 2)
        orig_in = rng.integers(0, 1000, (B, n)).astype(np.int32) if trial % 3 == 0 else None
        ki, nl, ngp, oo = oracle.ltp_prune(s, vl, gp, theta, kg, orig_in)
        ref = brute_prune(s, vl, gp, theta, kg, orig_in)
        for b, (kept, ng, orig) in enumerate(ref):
            assert nl[b] == len(kept)
            assert list(ki[b, :nl[b]]) == kept and np.all(ki[b, nl[b]:] == -1)
            assert list(ngp[b, :len(ng)]) == ng and np.all(ngp[b, len(ng):] == -1)
            assert list(oo[b, :nl[b]]) == orig and np.all(oo[b, nl[b]:] == -1)


def _topk_inputs(rng, B=4, n=60, G=3, levels=None):
    """Scores (optionally quantised to a few levels, so that ties are common), lengths, global positions."""
    s = rng.random((B, n)).astype(np.float32) * 0.05
    if levels:
        s = (np.floor(s / 0.05 * levels) / levels * 0.05).astype(np.float32)
    vl = rng.integers(0, n + 1, B).astype(np.int32)
    gp = np.full((B, G), -1, np.int32)
    for b in range(B):
        g = rng.choice(max(vl[b], 1), size=min(G, vl[b]), replace=False) if vl[b] else []
        gp[b, :len(g)] = np.sort(g)
    return s, vl, gp


def check_topk_rank_invariants():
    """Kept candidates: exactly ceil(ratio * C) of them; no dropped candidate scores above a kept one; at the
    boundary score the kept ones precede the dropped ones; globals kept; survivors in order."""
    rng = np.random.default_rng(11)
    for trial in range(40):
        s, vl, gp = _topk_inputs(rng, levels=(4 if trial % 2 else None))
        ratio = float(rng.choice([0.0, 0.1, 0.25, 0.5, 0.77, 1.0]))
        kg = int(trial % 3 != 0)
        ki, nl, ngp, _ = oracle.topk_prune(s, vl, gp, ratio, kg)
        for b in range(s.shape[0]):
            L = int(vl[b])
            g = set(int(p) for p in gp[b] if 0 <= p < L)
            kept = ki[b, :nl[b]].tolist()
            assert kept == sorted(set(kept)) and all(0 <= k < L for k in kept)
            cand = [k for k in range(L) if not (kg and k in g)]
            K = math.ceil(np.float64(np.float32(ratio)) * len(cand)) if ratio > 0 else 0
            kc = [k for k in kept if k in cand]
            dropped = [k for k in cand if k not in set(kc)]
            assert len(kc) == min(K, len(cand))
            if kg:
                assert g <= set(kept)
            if kc and dropped:
                lo = min(s[b, k] for k in kc)
                assert max(s[b, k] for k in dropped) <= lo
                tie_kept = [k for k in kc if s[b, k] == lo]
                tie_dropped = [k for k in dropped if s[b, k] == lo]
                if tie_dropped:
                    assert max(tie_kept) < min(tie_dropped)


def check_topk_equals_threshold_rule():
    """When the cut falls in a gap of the scores, top-k keeps exactly what the (separately pinned) threshold
    rule keeps with a threshold inside that gap; ratio 1 keeps every valid token, ratio 0 only the globals."""
    rng = np.random.default_rng(12)
    for trial in range(30):
        s, vl, gp = _topk_inputs(rng, B=1)
        L = int(vl[0])
        g = set(int(p) for p in gp[0] if 0 <= p < L)
        cand = sorted((float(s[0, k]) for k in range(L) if k not in g), reverse=True)
        if len(cand) >= 2:
            K = int(rng.integers(1, len(cand)))
            if cand[K - 1] > cand[K]:
                theta = float(np.float32((cand[K - 1] + cand[K]) / 2))
                ratio = (K - 0.5) / len(cand)
                a = oracle.topk_prune(s, vl, gp, ratio, 1)
                t = oracle.ltp_prune(s, vl, gp, theta, 1)
                for x, y in zip(a, t):
                    assert np.array_equal(x, y)
        ki, nl, _, _ = oracle.topk_prune(s, vl, gp, 1.0, 1)
        assert nl[0] == L and list(ki[0, :L]) == list(range(L))
        ki, nl, _, _ = oracle.topk_prune(s, vl, gp, 0.0, 1)
        assert list(ki[0, :nl[0]]) == sorted(g)
        ki, nl, _, _ = oracle.topk_prune(s, vl, gp, 0.0, 0)
        assert nl[0] == 0


def check_prune_invariants():
    q, k, v, vl, gp, w = rand_case(400, n=64, B=3)
    _, _, s = run(q, k, v, vl, gp, w)
    s32 = s.astype(np.float32)
    prev = None
    for theta in (-1.0, 0.0, 0.005, 0.01, 0.02, 0.05, 0.2):
        ki, nl, ngp, _ = oracle.ltp_prune(s32, vl, gp, theta, 1)
        for b in range(3):
            kept = set(ki[b, :nl[b]].tolist())
            g = set(int(p) for p in gp[b] if 0 <= p < vl[b])
            assert g <= kept                                   # globals always kept
            assert list(ki[b, :nl[b]]) == sorted(kept)         # stable order
            if theta > 0:
                assert len(kept - g) < 1.0 / theta             # scores sum to one
            if theta < 0:
                assert nl[b] == vl[b]                          # keeps every valid token
            if prev is not None:
                assert kept <= prev[b]                         # nested as theta grows
        prev = [set(ki[b, :nl[b]].tolist()) for b in range(3)]


def check_mask_rule_golden():
    cases = json.load(open(os.path.join(GOLDEN, "mask_rule.json")))["cases"]
    for c in cases:
        s = np.array([[c["score"], 1.0]], np.float32)
        ki, nl, _, _ = oracle.ltp_prune(s, np.array([2], np.int32), np.full((1, 1), -1, np.int32),
                                        c["threshold"], 1)
        assert int(0 in ki[0, :nl[0]]) == c["mask"]


def check_gather_rows():
    rng = np.random.default_rng(9)
    src = rng.integers(0, 2 ** 16, (2, 10, 7), dtype=np.uint16)
    ki = np.array([[1, 4, 9] + [-1] * 7, [0, 2] + [-1] * 8], np.int32)
    nl = np.array([3, 2], np.int32)
    dst = oracle.gather_rows(src, ki, nl)
    assert np.array_equal(dst[0, :3], src[0, [1, 4, 9]]) and np.array_equal(dst[1, :2], src[1, [0, 2]])
    assert np.all(dst[0, 3:] == 0)


def _torch_bf16(x):
    return torch.from_numpy(np.asarray(x, np.float64)).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()


def check_bf16_rounding():
    rng = np.random.default_rng(11)
    x = (rng.standard_normal(5000) * np.exp(rng.uniform(-20, 20, 5000))).astype(np.float32).astype(np.float64)
    ours = np.array([oracle.round_bf16(t) for t in x])
    assert np.array_equal(ours, _torch_bf16(x))
    # ties go to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7
    assert oracle.round_bf16(1 + 2 ** -8) == 1.0
    assert oracle.round_bf16(1 + 3 * 2 ** -8) == 1 + 2 ** -6
    assert oracle.round_bf16(-(1 + 2 ** -8)) == -1.0


def _ref_layer(x, wqkv, wo, vl, gp, H, alpha, theta, eps, w1=None, w2=None):
    """Library composition for dense windows: numpy matmul, torch SDPA, torch layer_norm, torch bf16, and for
    the feed-forward block torch's exact GELU."""
    B, n, D = x.shape
    d = D // H
    qkv = _torch_bf16(x @ wqkv)
    q, k, v = (qkv[..., i * D:(i + 1) * D].reshape(B, n, H, d) for i in range(3))
    y = np.zeros_like(x)
    kept_all, nl = [], []
    for b in range(B):
        L = int(vl[b])
        Q, K, V = (torch.from_numpy(t[b:b + 1, :L]).permute(0, 2, 1, 3) for t in (q, k, v))
        O = torch.nn.functional.scaled_dot_product_attention(Q, K, V, scale=alpha)
        P = torch.softmax(alpha * Q @ K.transpose(-1, -2), -1)
        s = (P.sum(2).mean(1)[0] / L).numpy().astype(np.float32)
        g = [int(p) for p in gp[b] if 0 <= p < L]
        kept = [j for j in range(L) if s[j] > np.float32(theta) or j in g]
        O = _torch_bf16(O.permute(0, 2, 1, 3).reshape(L, D).numpy())
        t = torch.from_numpy(x[b, :L] + O @ wo)
        yy = _torch_bf16(torch.nn.functional.layer_norm(t, (D,), eps=eps).numpy())
        if w1 is not None:
            h = _torch_bf16(torch.nn.functional.gelu(torch.from_numpy(yy @ w1), approximate="none").numpy())
            yy = _torch_bf16(torch.nn.functional.layer_norm(torch.from_numpy(yy + h @ w2), (D,), eps=eps).numpy())
        y[b, :len(kept)] = yy[kept]
        kept_all.append(kept)
        nl.append(len(kept))
    return y, kept_all, nl


def stack_case(seed=500, B=2, n=24, H=2, d=8):
    rng = np.random.default_rng(seed)
    D = H * d
    bf = _torch_bf16
    x = bf(rng.standard_normal((B, n, D)))
    wqkv = bf(rng.standard_normal((D, 3 * D)) * 0.3)
    wo = bf(rng.standard_normal((D, D)) * 0.3)
    vl = np.array([n, n - 7][:B], np.int32)
    gp = np.array([[0], [3]][:B], np.int32)
    return x, wqkv, wo, vl, gp, H


def check_encoder_layer_against_libraries():
    x, wqkv, wo, vl, gp, H = stack_case()
    n = x.shape[1]
    # scores here are about 1/L (~0.04-0.06): the threshold prunes some, keeps some
    for theta in (-1.0, 0.045):
        y, ki, nl, ngp, sc = oracle.encoder_layer(x, wqkv, wo, vl, gp, H, 2 * n, 0.6, theta)
        ry, rkept, rnl = _ref_layer(x, wqkv, wo, vl, gp, H, 0.6, theta, 1e-5)
        assert list(nl) == rnl
        for b in range(x.shape[0]):
            assert list(ki[b, :nl[b]]) == rkept[b]
        diff = np.abs(y - ry)
        ulp = np.maximum(np.abs(ry), 1e-30) * 2.0 ** -7
        assert np.all(diff <= ulp)                    # at most one bf16 step apart ...
        assert np.mean(diff == 0) > 0.995             # ... and nearly all identical


def _ffn_weights(seed, D, F=None):
    rng = np.random.default_rng(seed)
    F = F or 4 * D
    return _torch_bf16(rng.standard_normal((D, F)) * 0.3), _torch_bf16(rng.standard_normal((F, D)) * 0.3)


def check_ffn_layer_against_libraries():
    """Full layer (attention, prune, Wo + LN, GELU feed-forward + LN) against the library composition."""
    x, wqkv, wo, vl, gp, H = stack_case(503)
    n, D = x.shape[1], x.shape[2]
    w1, w2 = _ffn_weights(7, D)
    for theta in (-1.0, 0.045):
        y, ki, nl, ngp, sc = oracle.encoder_layer(x, wqkv, wo, vl, gp, H, 2 * n, 0.6, theta, w1=w1, w2=w2)
        ry, rkept, rnl = _ref_layer(x, wqkv, wo, vl, gp, H, 0.6, theta, 1e-5, w1, w2)
        assert list(nl) == rnl
        diff = np.abs(y - ry)
        ulp = np.maximum(np.abs(ry), 1e-30) * 2.0 ** -7
        assert np.mean(diff <= ulp) > 0.998           # one bf16 step, except where a step upstream moved it
        assert np.mean(diff == 0) > 0.98


def check_ffn_zero_output_weights():
    """W2 = 0: the feed-forward block adds nothing, so the layer is LayerNorm of the attention-only output."""
    x, wqkv, wo, vl, gp, H = stack_case(504)
    D = x.shape[2]
    w1, _ = _ffn_weights(8, D)
    y, ki, nl, _, _ = oracle.encoder_layer(x, wqkv, wo, vl, gp, H, 6, 0.6, 0.04, w1=w1, w2=np.zeros((4 * D, D)))
    y0, ki0, nl0, _, _ = oracle.encoder_layer(x, wqkv, wo, vl, gp, H, 6, 0.6, 0.04)
    assert np.array_equal(ki, ki0) and np.array_equal(nl, nl0)
    ref = _torch_bf16(torch.nn.functional.layer_norm(torch.from_numpy(y0), (D,), eps=1e-5).numpy())
    for b in range(x.shape[0]):
        assert np.array_equal(y[b, :nl[b]], ref[b, :nl[b]])
        assert np.all(y[b, nl[b]:] == 0)


def check_full_stack_composition():
    """Full stack with per-layer windows = its layers applied in turn."""
    x, wqkv, wo, vl, gp, H = stack_case(505)
    n, D = x.shape[1], x.shape[2]
    th = [0.0, 0.05, 0.06]
    wins = [2, 6, 2 * n]
    wq = [wqkv, wqkv[:, ::-1].copy(), wqkv * 0.5]
    wo_ = [wo, wo.T.copy(), wo]
    f1, f2 = zip(*[_ffn_weights(20 + l, D, 3 * D) for l in range(3)])
    y, fl, oi, kpl = oracle.encoder_stack(x, wq, wo_, vl, gp, H, wins, 0.6, th, w1_list=f1, w2_list=f2)
    cur, cl, cg = x, vl, gp
    orig = np.where(np.arange(n)[None, :] < vl[:, None], np.arange(n)[None, :], -1)
    for l in range(3):
        cur, ki, cl, cg, _ = oracle.encoder_layer(cur, wq[l], wo_[l], cl, cg, H, wins[l], 0.6, th[l], w1=f1[l],
                                                  w2=f2[l])
        orig = np.where(ki >= 0, np.take_along_axis(orig, np.maximum(ki, 0), 1), -1)
        assert list(kpl[l]) == list(cl)
    assert np.array_equal(y, cur) and list(fl) == list(cl) and np.array_equal(oi, orig)


def check_layernorm_statistics():
    x, wqkv, wo, vl, gp, H = stack_case(501)
    y, ki, nl, _, _ = oracle.encoder_layer(x, wqkv, wo, vl, gp, H, 6, 0.6, -1.0)
    for b in range(x.shape[0]):
        rows = y[b, :nl[b]]
        assert np.all(np.abs(rows.mean(1)) < 2e-2)
        assert np.all(np.abs(rows.var(1) - 1.0) < 3e-2)


def check_stack_composition():
    """Stack = layers applied in turn; theta = -1 keeps everything (identity orig_idx)."""
    x, wqkv, wo, vl, gp, H = stack_case(502)
    n = x.shape[1]
    th = [0.0, 0.05, 0.06]
    w1 = [wqkv, wqkv[:, ::-1].copy(), wqkv * 0.5]
    w2 = [wo, wo.T.copy(), wo]
    y, fl, oi, kpl = oracle.encoder_stack(x, w1, w2, vl, gp, H, 6, 0.6, th)
    cur, cl, cg = x, vl, gp
    orig = np.where(np.arange(n)[None, :] < vl[:, None], np.arange(n)[None, :], -1)
    for l in range(3):
        cur, ki, cl, cg, _ = oracle.encoder_layer(cur, w1[l], w2[l], cl, cg, H, 6, 0.6, th[l])
        orig = np.where(ki >= 0, np.take_along_axis(orig, np.maximum(ki, 0), 1), -1)
        assert list(kpl[l]) == list(cl)
    assert np.array_equal(y, cur) and list(fl) == list(cl) and np.array_equal(oi, orig)
    y0, fl0, oi0, _ = oracle.encoder_stack(x, w1, w2, vl, gp, H, 6, 0.6, [-1.0] * 3)
    assert list(fl0) == list(vl)
    for b in range(2):
        assert list(oi0[b, :vl[b]]) == list(range(vl[b]))


def check_paper_threshold_schedule():
    g = json.load(open(os.path.join(GOLDEN, "paper_threshold_schedule.json")))
    sched = si.paper_threshold_schedule(g["final_threshold"], g["n_layers"])
    for layer, val in g["printed"].items():
        assert abs(sched[int(layer) - 1] - val) < 1e-15


# ------------------------------------------------- soft pruning (training) --
def _soft_case(seed, T=0.02):
    """A small case whose threshold sits at the median score, so that most masks are on the sigmoid's slope."""
    q, k, v, vl, gp, window = rand_case(seed, B=2, n=20, H=2, d=6, G=2)
    alpha = 0.35
    _, _, s, _, _ = oracle.soft_prune_forward(q, k, v, vl, gp, window, alpha, 0.0, 1.0)
    theta = float(np.median(s[s > 0]))
    rng = np.random.default_rng(seed + 1)
    dy = rng.standard_normal(q.shape)
    dm = rng.standard_normal(s.shape)
    return q, k, v, vl, gp, window, alpha, theta, T, dy, dm, rng


def check_soft_backward_finite_differences():
    """Central differences of the forward's loss sum(y * dy) + sum(mask * dmask) against the backward."""
    for seed, use_dm in ((700, True), (701, False)):
        q, k, v, vl, gp, window, alpha, theta, T, dy, dm, rng = _soft_case(seed)
        dm = dm if use_dm else None

        def loss(x, th):
            _, _, _, m, y = oracle.soft_prune_forward(x[0], x[1], x[2], vl, gp, window, alpha, th, T)
            return float((y * dy).sum() + ((m * dm).sum() if dm is not None else 0.0))

        grads = oracle.soft_prune_backward(q, k, v, vl, gp, window, alpha, theta, T, dy, dm)
        h = 1e-6
        B, n, H, d = q.shape
        for which in range(3):
            for _ in range(8):
                b = int(rng.integers(B))
                idx = (b, int(rng.integers(vl[b])), int(rng.integers(H)), int(rng.integers(d)))
                xp = [q.copy(), k.copy(), v.copy()]
                xm = [q.copy(), k.copy(), v.copy()]
                xp[which][idx] += h
                xm[which][idx] -= h
                fd = (loss(xp, theta) - loss(xm, theta)) / (2 * h)
                an = grads[which][idx]
                assert abs(fd - an) <= 1e-5 * abs(an) + 1e-7, (seed, which, idx, fd, an)
        fd = (loss([q, k, v], theta + h) - loss([q, k, v], theta - h)) / (2 * h)
        assert abs(fd - grads[3]) <= 1e-5 * abs(grads[3]) + 1e-6, (seed, fd, grads[3])
        for b in range(B):  # padding tokens are neither queries nor keys
            for g in grads[:3]:
                assert np.all(g[b, vl[b]:] == 0.0)


def _torch_soft_loss(q, k, v, vl, gp, window, alpha, theta, T, dy, dm, keep_global=1):
    """The soft-pruned layer as dense masked attention in torch (float64); autograd gives its backward."""
    B, n, H, d = q.shape
    r = window // 2
    loss = q.new_zeros(())
    for b in range(B):
        L = int(vl[b])
        gf = np.zeros(n, bool)
        for p in gp[b]:
            if 0 <= p < L:
                gf[p] = True
        A = torch.from_numpy(allowed_matrix(n, L, r, gf)[:L, :L])
        cols, outs = [], []
        for h in range(H):
            S = alpha * q[b, :L, h] @ k[b, :L, h].T
            P = torch.softmax(S.masked_fill(~A, float("-inf")), dim=1)
            cols.append(P.sum(0))
            outs.append(P @ v[b, :L, h])
        s = torch.stack(cols).sum(0) / (H * L)
        gt = torch.from_numpy(gf[:L])
        m = torch.sigmoid((s - theta) / T)
        if keep_global:
            m = torch.where(gt, torch.ones_like(m), m)
        out = torch.stack(outs, 1)  # [L, H, d]
        loss = loss + (m[:, None, None] * out * dy[b, :L]).sum() + (m * dm[b, :L]).sum()
    return loss


def check_soft_backward_against_autograd():
    for seed, kg in ((710, 1), (711, 0), (712, 1)):
        q, k, v, vl, gp, window, alpha, theta, T, dy, dm, _ = _soft_case(seed)
        dq, dk, dv, dth = oracle.soft_prune_backward(q, k, v, vl, gp, window, alpha, theta, T, dy, dm,
                                                     keep_global=kg)
        tq, tk, tv = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v))
        tth = torch.tensor(theta, dtype=torch.float64, requires_grad=True)
        loss = _torch_soft_loss(tq, tk, tv, vl, gp, window, alpha, tth, T, torch.from_numpy(dy),
                                torch.from_numpy(dm), kg)
        loss.backward()
        for ours, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
            ref = ref.numpy()
            assert np.allclose(ours, ref, rtol=1e-9, atol=1e-11), float(np.abs(ours - ref).max())
        assert abs(dth - float(tth.grad)) <= 1e-9 * abs(dth) + 1e-11, (dth, float(tth.grad))


def check_soft_mask_limits():
    """Temperature to 0: the soft mask becomes the binarised mask of the hard rule (Sec. 4.2.2 step 2); the
    threshold far below every score: the mask is 1 and y is the attention output."""
    q, k, v, vl, gp, window, alpha, theta, _, _, _, _ = _soft_case(720)
    out, _, s, m, y = oracle.soft_prune_forward(q, k, v, vl, gp, window, alpha, theta, 1e-12)
    B, n = s.shape
    for b in range(B):
        g = {int(p) for p in gp[b] if 0 <= p < vl[b]}
        for t in range(n):
            hard = t < vl[b] and (s[b, t] > theta or t in g)
            if t < vl[b] and t not in g and abs(s[b, t] - theta) < 1e-9:
                continue
            assert m[b, t] == (1.0 if hard else 0.0), (b, t, m[b, t], s[b, t], theta)
    assert np.array_equal(y, out * m[:, :, None, None])
    out2, _, _, m2, y2 = oracle.soft_prune_forward(q, k, v, vl, gp, window, alpha, -1e6, 0.01)
    valid = np.arange(n)[None, :] < vl[:, None]
    assert np.all(m2[valid] == 1.0) and np.all(m2[~valid] == 0.0)
    assert np.array_equal(y2, out2)


def check_soft_backward_error_scales():
    """The error scales of the backward (the chain on magnitudes) dominate the gradients, and bound the first-order
    change of every gradient element when every element of dy is perturbed by a relative delta of random sign:
    dy enters the chain linearly (through m * dy and through the mask gradient sum(dy * out)), so that change is at
    most delta times the scale."""
    for seed, kg in ((730, 1), (731, 0)):
        q, k, v, vl, gp, window, alpha, theta, T, dy, dm, rng = _soft_case(seed)
        dq, dk, dv, dth, mq, mk, mv, mth = oracle.soft_prune_backward(q, k, v, vl, gp, window, alpha, theta, T, dy,
                                                                      dm, keep_global=kg, scales=True)
        for g, m in ((dq, mq), (dk, mk), (dv, mv)):
            assert np.all(np.abs(g) <= m * (1 + 1e-12) + 1e-300)
        assert abs(dth) <= mth * (1 + 1e-12)
        delta = 1e-7
        sign = rng.choice([-1.0, 1.0], size=dy.shape)
        sgn_m = rng.choice([-1.0, 1.0], size=dm.shape)
        # dmask perturbed too: its magnitude is part of the scales
        g2 = oracle.soft_prune_backward(q, k, v, vl, gp, window, alpha, theta, T, dy * (1 + delta * sign),
                                        dm * (1 + delta * sgn_m), keep_global=kg)
        for g, gp2, m in ((dq, g2[0], mq), (dk, g2[1], mk), (dv, g2[2], mv)):
            assert np.all(np.abs(gp2 - g) <= delta * m * (1 + 1e-6) + 1e-15 * np.abs(g).max()), \
                float((np.abs(gp2 - g) / np.maximum(delta * m, 1e-300)).max())
        assert abs(g2[3] - dth) <= delta * mth * (1 + 1e-6) + 1e-12 * abs(dth)
        # a tighter scale would fail: for dv (a plain sum of P * m * dy) the scale is reached when all signs agree
        g3 = oracle.soft_prune_backward(q, k, v, vl, gp, window, alpha, theta, T, dy * (1 + delta * np.sign(dy)),
                                        dm, keep_global=kg)
        b = 0
        L = int(vl[b])
        ratio = np.abs(g3[2][b, :L] - dv[b, :L]) / np.maximum(delta * mv[b, :L], 1e-300)
        assert ratio.max() > 0.5, float(ratio.max())


SOFT_CHECKS = [check_soft_backward_finite_differences, check_soft_backward_against_autograd,
               check_soft_mask_limits, check_soft_backward_error_scales]

ATTENTION_CHECKS = [check_brute_force, check_causal_brute_force, check_causal_dense_is_library_causal_attention,
                    check_window_covers_sequence_is_dense, check_all_global_is_dense,
                    check_zero_window_no_global, check_constant_values, check_zero_queries_rational_scores,
                    check_score_invariants, check_reflection_symmetry, check_head_permutation,
                    check_sec55_example_structure, check_padding_is_invisible]
PRUNE_CHECKS = [check_prune_brute_force, check_prune_invariants, check_mask_rule_golden, check_gather_rows,
                check_topk_rank_invariants, check_topk_equals_threshold_rule]
STACK_CHECKS = [check_bf16_rounding, check_encoder_layer_against_libraries, check_layernorm_statistics,
                check_stack_composition, check_ffn_layer_against_libraries, check_ffn_zero_output_weights,
                check_full_stack_composition]
ALL_CHECKS = ATTENTION_CHECKS + PRUNE_CHECKS + STACK_CHECKS + SOFT_CHECKS + [check_paper_threshold_schedule]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__[6:])
def test_pin(check):
    check()
