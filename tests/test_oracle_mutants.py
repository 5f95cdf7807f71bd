"""Plant plausible mistakes in copies of the oracle (CPU only) and show that the
pins in test_oracle_pins.py catch every one of them.

Each mutant is a textual edit of sc_oracle.cpp compiled to a temporary library;
the pins then run against it and at least one must fail.
"""
import ctypes
import os
import subprocess

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "sc_oracle.cpp")

MUTANTS = [
    ("window off by one", "std::abs(i - j) <= r ||", "std::abs(i - j) < r ||"),
    ("global columns dropped", "|| is_global[i] || is_global[j]", "|| is_global[i]"),
    ("global rows dropped", "|| is_global[i] || is_global[j]", "|| is_global[j]"),
    ("scores divided by padded length", "acc / ((double)H * L)", "acc / ((double)H * n)"),
    ("column sum credited to the query", "colsum[nbr[t]] += p;", "colsum[i] += p;"),
    ("softmax sum without the max shift", "z += std::exp(s[t] - m);", "z += std::exp(s[t]);"),
    ("softmax scale ignored", "s[t] = alpha * acc;", "s[t] = acc;"),
    ("lse without the max", "lse[i] = m + std::log(z);", "lse[i] = std::log(z);"),
    ("padding row attends", "if (i >= L) {  // padding query", "if (i > L) {  // padding query"),
    ("non-strict mask", "scores[(long)b * n + k] > threshold", "scores[(long)b * n + k] >= threshold"),
    ("globals kept regardless of flag", "(keep_global && g[k])", "(g[k])"),
    ("globals not renumbered", "new_global_pos[(long)b * G + gc++] = new_index[p];",
     "new_global_pos[(long)b * G + gc++] = p;"),
    ("orig index not composed", "orig_in[(long)b * n + src]", "orig_in[(long)b * n + j]"),
    ("bf16 rounding truncates", "std::nearbyint(x / ulp) * ulp", "std::trunc(x / ulp) * ulp"),
    ("k and v projections swapped", "kv[row * D + j] = round_bf16(acc[D + j]);",
     "kv[row * D + j] = round_bf16(acc[2 * D + j]);"),
    ("attention output not stored as bf16", "for (auto& e : o) e = round_bf16(e);", ""),
    ("residual dropped", "t[c] = x[src * D + c];", "t[c] = 0.0;"),
    ("unbiased variance", "var /= (double)D;", "var /= (double)(D - 1);"),
    ("value of the query used", "const double* vj = v + (long)nbr[t] * ld;", "const double* vj = v + (long)i * ld;"),
    ("top-k ties to the higher index", "std::stable_sort(cand.begin()",
     "std::reverse(cand.begin(), cand.end());\n    std::stable_sort(cand.begin()"),
    ("top-k count rounded down", "(long)std::ceil(prod)", "(long)std::floor(prod)"),
    ("top-k counts kept globals as candidates", "      else\n        cand.push_back(k);", "      cand.push_back(k);"),
    ("GELU replaced by ReLU", "return 0.5 * v * (1.0 + std::erf(v / std::sqrt(2.0)));", "return v > 0.0 ? v : 0.0;"),
    ("feed-forward residual dropped", "for (long c = 0; c < D; ++c) t[c] = x1[c];", "for (long c = 0; c < D; ++c) t[c] = 0.0;"),
    ("feed-forward hidden not stored as bf16", "h[f] = round_bf16(gelu(h[f]));", "h[f] = gelu(h[f]);"),
    ("causal query sees the future", "const int jend = causal ? std::min(i + 1, L) : L;", "const int jend = L;"),
    ("causal global rows see the future", "const int jend = causal ? std::min(i + 1, L) : L;",
     "const int jend = causal && !is_global[i] ? std::min(i + 1, L) : L;"),
    ("per-layer window ignored", "int rc = encoder_layer(B, n, H, d, windows[l],", "int rc = encoder_layer(B, n, H, d, windows[0],"),
    ("soft mask: score gradient dropped", "gs[t] = ds / ((double)H * L);", "gs[t] = 0.0;"),
    ("soft mask: score gradient over the padded length", "gs[t] = ds / ((double)H * L);",
     "gs[t] = ds / ((double)H * n);"),
    ("soft mask: sigmoid derivative missing a factor", "const double ds = dm * mask[t] * (1.0 - mask[t]) / T;",
     "const double ds = dm * mask[t] / T;"),
    ("soft mask: temperature ignored in the backward", "const double ds = dm * mask[t] * (1.0 - mask[t]) / T;",
     "const double ds = dm * mask[t] * (1.0 - mask[t]);"),
    ("soft mask: threshold gradient sign", "dth -= ds;", "dth += ds;"),
    ("soft mask: output gradient not masked", "dout[t * D + c] = mask[t] * dy[t * D + c];",
     "dout[t * D + c] = dy[t * D + c];"),
    ("soft mask: softmax backward without the row term", "const double dsij = p[t] * (dp[t] - rowdot);",
     "const double dsij = p[t] * dp[t];"),
    ("soft mask: key gradient from the key", "dkh[(long)j * D + c] += alpha * dsij * qh[(long)i * D + c];",
     "dkh[(long)j * D + c] += alpha * dsij * kh[(long)i * D + c];"),
    ("soft mask: value gradient transposed", "dvh[(long)j * D + c] += p[t] * doh[(long)i * D + c];",
     "dvh[(long)i * D + c] += p[t] * doh[(long)j * D + c];"),
    ("soft mask: global tokens masked softly", "if (k < L) m = (keep_global && g[k]) ? 1.0 :",
     "if (k < L) m = false ? 1.0 :"),
]


def build_mutant(tmp_path, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    path = tmp_path / "mut.cpp"
    path.write_text(src.replace(old, new, 1))
    so = tmp_path / "libmut.so"
    subprocess.run(["g++", "-std=c++17", "-O1", "-fopenmp", "-fPIC", "-shared", str(path), "-o", str(so)],
                   check=True)
    return str(so)


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, monkeypatch, name, old, new):
    so = build_mutant(tmp_path, old, new)
    saved = oracle._lib
    oracle._lib = None
    monkeypatch.setattr(oracle, "_LIB", so)
    try:
        oracle.lib()
        caught = []
        for check in pins.ALL_CHECKS:
            try:
                check()
            except AssertionError:
                caught.append(check.__name__)
        assert caught, f"no pin caught mutant '{name}'"
    finally:
        oracle._lib = saved
