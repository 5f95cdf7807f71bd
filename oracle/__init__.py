"""CPU oracle for the sparse-attention + learned-token-pruning path (TEST INFRASTRUCTURE).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never does, and this package imports nothing from it.

The arithmetic lives in ``sc_oracle.cpp`` (plain C++17, double precision,
OpenMP over (sequence, head)); this module only builds and marshals it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sc_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")
_SAN_LIB = os.path.join(_HERE, "liboracle_san.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["g++", "-std=c++17", "-O2", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared", _SRC,
                        "-o", tmp], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized() -> str:
    """Compile the oracle with AddressSanitizer and UndefinedBehaviorSanitizer (host code only; every UB report
    aborts).  Load it by setting SC_ORACLE_LIB to the returned path, with the sanitizer runtimes preloaded."""
    tmp = _SAN_LIB + ".tmp"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fno-fast-math", "-fopenmp",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fPIC", "-shared", _SRC,
                    "-o", tmp], check=True)
    os.replace(tmp, _SAN_LIB)
    return _SAN_LIB


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("SC_ORACLE_LIB") or _LIB
        if path == _LIB and not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(path)
        i32p = ctypes.POINTER(ctypes.c_int32)
        f64p = ctypes.POINTER(ctypes.c_double)
        f32p = ctypes.POINTER(ctypes.c_float)
        ci, cd, cf, vp, cl = ctypes.c_int, ctypes.c_double, ctypes.c_float, ctypes.c_void_p, ctypes.c_long
        L.orc_round_bf16.argtypes = [cd]
        L.orc_round_bf16.restype = cd
        L.orc_sparse_attention.argtypes = [ci, ci, ci, ci, ci, ci, i32p, i32p, cd, f64p, f64p, f64p, f64p, f64p,
                                           f64p, f64p, ci]
        L.orc_sparse_attention_causal.argtypes = L.orc_sparse_attention.argtypes
        L.orc_ltp_prune.argtypes = [ci, ci, ci, i32p, i32p, f32p, cf, ci, i32p, i32p, i32p, i32p, i32p]
        L.orc_topk_prune.argtypes = [ci, ci, ci, i32p, i32p, f32p, cf, ci, i32p, i32p, i32p, i32p, i32p]
        L.orc_gather_rows.argtypes = [ci, ci, cl, vp, vp, i32p, i32p]
        L.orc_encoder_layer.argtypes = [ci, ci, ci, ci, ci, ci, i32p, i32p, cd, f64p, f64p, f64p, cf, ci, cd, f64p,
                                        i32p, i32p, i32p, f32p, ci]
        L.orc_encoder_stack.argtypes = [ci, ci, ci, ci, ci, ci, i32p, i32p, cd, ci, f64p, f64p, f64p, f32p, ci, cd,
                                        f64p, i32p, i32p, i32p, ci]
        L.orc_encoder_layer_ffn.argtypes = [ci, ci, ci, ci, ci, ci, i32p, i32p, cd, f64p, f64p, f64p, f64p, f64p, ci,
                                            cf, ci, cd, f64p, i32p, i32p, i32p, f32p, ci]
        L.orc_encoder_stack_ffn.argtypes = [ci, ci, ci, ci, i32p, ci, i32p, i32p, cd, ci, f64p, f64p, f64p, f64p,
                                            f64p, ci, f32p, ci, cd, f64p, i32p, i32p, i32p, ci]
        L.orc_soft_prune_forward.argtypes = [ci, ci, ci, ci, ci, ci, i32p, i32p, cd, f64p, f64p, f64p, cd, cd, ci,
                                             f64p, f64p, f64p, f64p, f64p, ci]
        L.orc_soft_prune_backward.argtypes = [ci, ci, ci, ci, ci, ci, i32p, i32p, cd, f64p, f64p, f64p, cd, cd, ci,
                                              f64p, f64p, f64p, f64p, f64p, f64p, f64p, f64p, f64p, f64p, ci]
        for f in ("orc_sparse_attention", "orc_sparse_attention_causal", "orc_ltp_prune", "orc_topk_prune",
                  "orc_gather_rows", "orc_encoder_layer", "orc_encoder_stack", "orc_encoder_layer_ffn",
                  "orc_encoder_stack_ffn", "orc_soft_prune_forward", "orc_soft_prune_backward"):
            getattr(L, f).restype = ci
        _lib = L
    return _lib


def _p(a, ct):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ct))


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def default_threads() -> int:
    for var in ("SC_ORACLE_THREADS", "OMP_NUM_THREADS"):
        v = os.environ.get(var, "")
        if v.isdigit() and int(v) > 0:
            return int(v)
    return os.cpu_count() or 1


def round_bf16(x: float) -> float:
    return lib().orc_round_bf16(float(x))


def sparse_attention(q, k, v, valid_len, global_pos, window, alpha, want_colsum=False, nthreads=None, causal=False):
    """q, k, v: [B, n, H, d] doubles.  Returns (out, lse, scores[, colsum]).  causal: keys after the query are
    not attended."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, n, H, d = q.shape
    gp = _i32(global_pos).reshape(B, -1)
    G = gp.shape[1]
    vl = _i32(valid_len)
    out = np.empty_like(q)
    lse = np.empty((B, H, n))
    scores = np.empty((B, n))
    colsum = np.empty((B, H, n)) if want_colsum else None
    fn = lib().orc_sparse_attention_causal if causal else lib().orc_sparse_attention
    rc = fn(B, n, H, d, int(window), G, _p(gp, ctypes.c_int32), _p(vl, ctypes.c_int32),
                                    float(alpha), _p(q, ctypes.c_double), _p(k, ctypes.c_double),
                                    _p(v, ctypes.c_double), _p(out, ctypes.c_double), _p(lse, ctypes.c_double),
                                    _p(scores, ctypes.c_double), _p(colsum, ctypes.c_double),
                                    nthreads or default_threads())
    assert rc == 0, rc
    return (out, lse, scores, colsum) if want_colsum else (out, lse, scores)


def soft_prune_forward(q, k, v, valid_len, global_pos, window, alpha, theta, temperature, keep_global=1,
                       nthreads=None):
    """LTP soft pruning, training form.  Returns (out, lse, scores, mask [B, n], y [B, n, H, d] = mask * out)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, n, H, d = q.shape
    gp = _i32(global_pos).reshape(B, -1)
    vl = _i32(valid_len)
    out, y = np.empty_like(q), np.empty_like(q)
    lse, scores, mask = np.empty((B, H, n)), np.empty((B, n)), np.empty((B, n))
    c = ctypes.c_double
    rc = lib().orc_soft_prune_forward(B, n, H, d, int(window), gp.shape[1], _p(gp, ctypes.c_int32),
                                      _p(vl, ctypes.c_int32), float(alpha), _p(q, c), _p(k, c), _p(v, c),
                                      float(theta), float(temperature), int(keep_global), _p(out, c), _p(lse, c),
                                      _p(scores, c), _p(mask, c), _p(y, c), nthreads or default_threads())
    assert rc == 0, rc
    return out, lse, scores, mask, y


def soft_prune_backward(q, k, v, valid_len, global_pos, window, alpha, theta, temperature, dy, dmask=None,
                        keep_global=1, nthreads=None, scales=False):
    """Backward of soft_prune_forward for dL/dy = dy [B, n, H, d] and dL/dmask = dmask [B, n] (or None).
    Returns (dq, dk, dv, dtheta); with scales, also (mq, mk, mv, mtheta): the same chain on magnitudes, the
    error scale of each gradient element."""
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    B, n, H, d = q.shape
    gp = _i32(global_pos).reshape(B, -1)
    vl = _i32(valid_len)
    dm = _f64(dmask) if dmask is not None else None
    dq, dk, dv = np.empty_like(q), np.empty_like(q), np.empty_like(q)
    dth = np.zeros(1)
    mq, mk, mv, mth = (np.empty_like(q), np.empty_like(q), np.empty_like(q), np.zeros(1)) if scales else \
        (None, None, None, None)
    c = ctypes.c_double
    rc = lib().orc_soft_prune_backward(B, n, H, d, int(window), gp.shape[1], _p(gp, ctypes.c_int32),
                                       _p(vl, ctypes.c_int32), float(alpha), _p(q, c), _p(k, c), _p(v, c),
                                       float(theta), float(temperature), int(keep_global), _p(dy, c), _p(dm, c),
                                       _p(dq, c), _p(dk, c), _p(dv, c), _p(dth, c), _p(mq, c), _p(mk, c), _p(mv, c),
                                       _p(mth, c), nthreads or default_threads())
    assert rc == 0, rc
    if scales:
        return dq, dk, dv, float(dth[0]), mq, mk, mv, float(mth[0])
    return dq, dk, dv, float(dth[0])


def ltp_prune(scores32, valid_len, global_pos, threshold, keep_global=1, orig_in=None):
    """scores32: [B, n] float32.  Returns (keep_idx, new_len, new_global_pos, orig_out)."""
    return _prune(lib().orc_ltp_prune, scores32, valid_len, global_pos, threshold, keep_global, orig_in)


def topk_prune(scores32, valid_len, global_pos, keep_ratio, keep_global=1, orig_in=None):
    """Rank rule: keep ceil(keep_ratio * C) of the C candidates per sequence.  Returns as ltp_prune."""
    return _prune(lib().orc_topk_prune, scores32, valid_len, global_pos, keep_ratio, keep_global, orig_in)


def _prune(fn, scores32, valid_len, global_pos, value, keep_global, orig_in):
    s = np.ascontiguousarray(scores32, dtype=np.float32)
    B, n = s.shape
    gp = _i32(global_pos).reshape(B, -1)
    G = gp.shape[1]
    vl = _i32(valid_len)
    keep_idx = np.empty((B, n), np.int32)
    new_len = np.empty(B, np.int32)
    ngp = np.empty((B, G), np.int32)
    orig_out = np.empty((B, n), np.int32)
    oi = None if orig_in is None else _i32(orig_in)
    rc = fn(B, n, G, _p(gp, ctypes.c_int32), _p(vl, ctypes.c_int32), _p(s, ctypes.c_float), np.float32(value).item(),
            int(keep_global), _p(keep_idx, ctypes.c_int32), _p(new_len, ctypes.c_int32), _p(ngp, ctypes.c_int32),
            _p(oi, ctypes.c_int32), _p(orig_out, ctypes.c_int32))
    assert rc == 0
    return keep_idx, new_len, ngp, orig_out


def gather_rows(src, keep_idx, new_len, dst=None):
    """src: [B, n, ...] any dtype; rows >= new_len of dst are left as given (zeros if dst is None)."""
    src = np.ascontiguousarray(src)
    B, n = src.shape[:2]
    dst = np.zeros_like(src) if dst is None else dst
    row_bytes = src.nbytes // (B * n) if B * n else 0
    lib().orc_gather_rows(B, n, row_bytes, src.ctypes.data, dst.ctypes.data, _p(_i32(keep_idx), ctypes.c_int32),
                          _p(_i32(new_len), ctypes.c_int32))
    return dst


def encoder_layer(x, wqkv, wo, valid_len, global_pos, H, window, alpha, threshold, keep_global=1, ln_eps=1e-5,
                  nthreads=None, w1=None, w2=None):
    """x: [B, n, D] doubles (bf16 values).  Returns (y, keep_idx, new_len, new_global_pos, scores32).
    w1 [D, F], w2 [F, D]: the feed-forward block (None: attention-only layer)."""
    x = _f64(x)
    B, n, D = x.shape
    d = D // H
    gp = _i32(global_pos).reshape(B, -1)
    G = gp.shape[1]
    vl = _i32(valid_len)
    y = np.empty_like(x)
    keep_idx = np.empty((B, n), np.int32)
    new_len = np.empty(B, np.int32)
    ngp = np.empty((B, G), np.int32)
    sc = np.empty((B, n), np.float32)
    if w1 is not None:
        w1, w2 = _f64(w1), _f64(w2)
        rc = lib().orc_encoder_layer_ffn(
            B, n, H, d, int(window), G, _p(gp, ctypes.c_int32), _p(vl, ctypes.c_int32), float(alpha),
            _p(x, ctypes.c_double), _p(_f64(wqkv), ctypes.c_double), _p(_f64(wo), ctypes.c_double),
            _p(w1, ctypes.c_double), _p(w2, ctypes.c_double), int(w1.shape[1]), np.float32(threshold).item(),
            int(keep_global), float(ln_eps), _p(y, ctypes.c_double), _p(keep_idx, ctypes.c_int32),
            _p(new_len, ctypes.c_int32), _p(ngp, ctypes.c_int32), _p(sc, ctypes.c_float), nthreads or default_threads())
        assert rc == 0
        return y, keep_idx, new_len, ngp, sc
    rc = lib().orc_encoder_layer(B, n, H, d, int(window), G, _p(gp, ctypes.c_int32), _p(vl, ctypes.c_int32),
                                 float(alpha), _p(x, ctypes.c_double), _p(_f64(wqkv), ctypes.c_double),
                                 _p(_f64(wo), ctypes.c_double), np.float32(threshold).item(), int(keep_global),
                                 float(ln_eps), _p(y, ctypes.c_double), _p(keep_idx, ctypes.c_int32),
                                 _p(new_len, ctypes.c_int32), _p(ngp, ctypes.c_int32), _p(sc, ctypes.c_float),
                                 nthreads or default_threads())
    assert rc == 0
    return y, keep_idx, new_len, ngp, sc


def encoder_stack(x, wqkv_list, wo_list, valid_len, global_pos, H, window, alpha, thresholds, keep_global=1,
                  ln_eps=1e-5, nthreads=None, w1_list=None, w2_list=None):
    """Returns (y, final_len, orig_idx, kept_per_layer).  window: one int, or one per layer; w1_list / w2_list:
    the feed-forward blocks of the layers (None: attention-only layers)."""
    x = _f64(x)
    B, n, D = x.shape
    d = D // H
    nl = len(thresholds)
    gp = _i32(global_pos).reshape(B, -1)
    G = gp.shape[1]
    vl = _i32(valid_len)
    wq = _f64(np.stack(wqkv_list))
    wo = _f64(np.stack(wo_list))
    th = np.ascontiguousarray(thresholds, dtype=np.float32)
    y = np.empty_like(x)
    fl = np.empty(B, np.int32)
    oi = np.empty((B, n), np.int32)
    kpl = np.empty((nl, B), np.int32)
    if w1_list is not None or not np.isscalar(window):
        win = np.ascontiguousarray(np.broadcast_to(np.asarray(window, dtype=np.int32), (nl,)))
        assert w1_list is not None, "per-layer windows are part of the full stack"
        w1 = _f64(np.stack(w1_list))
        w2 = _f64(np.stack(w2_list))
        rc = lib().orc_encoder_stack_ffn(
            B, n, H, d, _p(win, ctypes.c_int32), G, _p(gp, ctypes.c_int32), _p(vl, ctypes.c_int32), float(alpha), nl,
            _p(x, ctypes.c_double), _p(wq, ctypes.c_double), _p(wo, ctypes.c_double), _p(w1, ctypes.c_double),
            _p(w2, ctypes.c_double), int(w1.shape[2]), _p(th, ctypes.c_float), int(keep_global), float(ln_eps),
            _p(y, ctypes.c_double), _p(fl, ctypes.c_int32), _p(oi, ctypes.c_int32), _p(kpl, ctypes.c_int32),
            nthreads or default_threads())
        assert rc == 0
        return y, fl, oi, kpl
    rc = lib().orc_encoder_stack(B, n, H, d, int(window), G, _p(gp, ctypes.c_int32), _p(vl, ctypes.c_int32),
                                 float(alpha), nl, _p(x, ctypes.c_double), _p(wq, ctypes.c_double),
                                 _p(wo, ctypes.c_double), _p(th, ctypes.c_float), int(keep_global), float(ln_eps),
                                 _p(y, ctypes.c_double), _p(fl, ctypes.c_int32), _p(oi, ctypes.c_int32),
                                 _p(kpl, ctypes.c_int32), nthreads or default_threads())
    assert rc == 0
    return y, fl, oi, kpl
