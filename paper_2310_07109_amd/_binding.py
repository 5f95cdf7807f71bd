"""ctypes binding of libsc.so (argument marshalling only)."""
from __future__ import annotations

import ctypes
import functools
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsc.so")
# the same library built with SC_DEBUG (device-side argument checks, a synchronisation per call)
_DEBUG_LIB_PATH = os.path.join(_HERE, "libsc_debug.so")

SC_OK, SC_EINVAL, SC_EUNSUPPORTED, SC_EWORKSPACE, SC_EHIP, SC_ENOSCRATCH = 0, -1, -2, -3, -4, -5
SC_NOALLOC_SCRATCH_BYTES = 16 << 20
# bits of sc_validate_desc's result
SC_VALID_LEN, SC_VALID_POS_RANGE, SC_VALID_POS_ORDER, SC_VALID_POS_UNUSED_FIRST = 1, 2, 4, 8
SC_F32, SC_BF16 = 0, 1
SC_SCORE_FROM_PARTIALS, SC_SCORE_FROM_BAND_PROBS = 0, 1

_lib = None
_debug_lib = None


class ScError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {sc_status_str(status)} ({status})")


class _Desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("n", ctypes.c_int32), ("H", ctypes.c_int32), ("d", ctypes.c_int32),
                ("window", ctypes.c_int32), ("G", ctypes.c_int32), ("global_pos", ctypes.c_void_p),
                ("valid_len", ctypes.c_void_p), ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("causal", ctypes.c_int32)]


def lib_path() -> str:
    return _LIB_PATH


def debug_lib_path() -> str:
    return _DEBUG_LIB_PATH


def load():
    """Load libsc.so; raises if it has not been built (no fallback path exists)."""
    global _lib
    if _lib is None:
        _lib = _open(_LIB_PATH)
    return _lib


def load_debug():
    """Load libsc_debug.so, the SC_DEBUG build (same entry points and signatures); raises if it is missing."""
    global _debug_lib
    if _debug_lib is None:
        _debug_lib = _open(_DEBUG_LIB_PATH)
    return _debug_lib


def _open(path):
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2310_07109_amd.build`")
    L = ctypes.CDLL(path)
    vp, sz, i32, f32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_float
    dp = ctypes.POINTER(_Desc)
    sig = {
        "sc_status_str": (ctypes.c_char_p, [i32]),
        "sc_score_partials_size": (sz, [dp]),
        "sc_band_probs_size": (sz, [dp]),
        "sc_window_attention_workspace_size": (sz, [dp]),
        "sc_window_attention": (i32, [dp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sc_window_attention_noalloc": (i32, [dp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "sc_ltp_score_workspace_size": (sz, [dp, i32]),
        "sc_ltp_score": (i32, [dp, i32, vp, vp, vp, sz, vp]),
        "sc_ltp_prune_compact_workspace_size": (sz, [dp]),
        "sc_ltp_prune_compact": (i32, [dp, vp, f32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sc_topk_prune_compact": (i32, [dp, vp, f32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sc_ltp_soft_mask": (i32, [dp, vp, f32, f32, i32, vp, vp, vp, vp]),
        "sc_ltp_soft_backward_workspace_size": (sz, [dp]),
        "sc_ltp_soft_backward": (i32, [dp, vp, vp, vp, vp, vp, vp, f32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sc_encoder_attn_stack_workspace_size": (sz, [dp, i32]),
        "sc_encoder_attn_stack": (i32, [dp, i32, vp, vp, vp, vp, i32, f32, vp, vp, vp, vp, vp, sz, vp]),
        "sc_encoder_stack_workspace_size": (sz, [dp, i32, i32]),
        "sc_encoder_stack": (i32, [dp, i32, vp, vp, vp, vp, vp, vp, i32, vp, i32, f32, vp, vp, vp, vp, vp, sz, vp]),
        "sc_validate_desc": (i32, [dp, vp, vp]),
        "sc_profile_window_kernel": (i32, [i32]),
        "sc_profile_window_kernel_read": (i32, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                                 ctypes.c_int64, ctypes.POINTER(ctypes.c_int64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


def sc_status_str(status: int) -> str:
    return load().sc_status_str(int(status)).decode()


def _check(status: int, where: str):
    if status != SC_OK:
        raise ScError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _tensor(t, name, dtype=None, shape=None, leading=None):
    """Checks a tensor argument before its pointer is marshalled: a contiguous CUDA tensor, of `dtype`, of
    exactly `shape` or with leading dimensions `leading`.  Returns it."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: expected a GPU tensor, got one on {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if leading is not None and tuple(t.shape[:len(leading)]) != tuple(leading):
        raise ValueError(f"{name}: expected leading dimensions {tuple(leading)}, got {tuple(t.shape)}")
    return t


def _min_bytes(t, name, nbytes):
    if t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name}: {t.numel() * t.element_size()} bytes, {nbytes} needed")
    return t


def _on_stream(fn):
    """Runs a wrapper with `stream` (when given) as torch's current stream, so that the outputs and workspaces
    it allocates belong to the stream its kernels are enqueued on: the caching allocator then never hands that
    memory to work on another stream while the kernels still use it."""
    @functools.wraps(fn)
    def run(*args, **kwargs):
        stream = kwargs.get("stream")
        if stream is None:
            return fn(*args, **kwargs)
        import torch
        with torch.cuda.stream(stream):
            return fn(*args, **kwargs)
    return run


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Desc:
    """Geometry of one attention layer (mirrors sc_attn_desc).

    valid_len: int32 device tensor [B]; global_pos: int32 device tensor [B, G] or None.
    """

    def __init__(self, B, n, H, window, valid_len, global_pos=None, softmax_scale=0.125, dtype=SC_BF16, d=64,
                 causal=False):
        self.B, self.n, self.H, self.d, self.window = int(B), int(n), int(H), int(d), int(window)
        self.valid_len = valid_len
        self.global_pos = global_pos
        self.G = 0 if global_pos is None else int(global_pos.shape[1])
        self.softmax_scale = float(softmax_scale)
        self.dtype = int(dtype)
        self.causal = int(bool(causal))

    def c(self) -> _Desc:
        return _Desc(self.B, self.n, self.H, self.d, self.window, self.G,
                     None if self.global_pos is None else self.global_pos.data_ptr(),
                     None if self.valid_len is None else self.valid_len.data_ptr(), self.softmax_scale, self.dtype,
                     self.causal)

    def torch_dtype(self):
        import torch
        return torch.bfloat16 if self.dtype == SC_BF16 else torch.float32


def _ws(nbytes, device):
    import torch
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def sc_score_partials_size(desc: Desc) -> int:
    return load().sc_score_partials_size(ctypes.byref(desc.c()))


def sc_band_probs_size(desc: Desc) -> int:
    return load().sc_band_probs_size(ctypes.byref(desc.c()))


def sc_window_attention_workspace_size(desc: Desc) -> int:
    return load().sc_window_attention_workspace_size(ctypes.byref(desc.c()))


def _opt(spec, make):
    """Output argument: True -> allocate, False/None -> absent, tensor -> use it."""
    if spec is True:
        return make()
    if spec is False or spec is None:
        return None
    return spec


@_on_stream
def sc_window_attention(desc: Desc, q, k, v, out=None, lse=True, score_partials=True, band_probs=False,
                        workspace=None, stream=None):
    """Returns (out, lse, score_partials, band_probs); absent outputs are None.

    lse / score_partials / band_probs: True (allocate), False (skip) or a preallocated tensor."""
    import torch
    L = load()
    cd = desc.c()
    shape = (desc.B, desc.n, desc.H, desc.d)
    for t, nm in ((q, "q"), (k, "k"), (v, "v")):
        _tensor(t, nm, desc.torch_dtype(), shape)
    dev = q.device
    out = torch.empty_like(q) if out is None else _tensor(out, "out", desc.torch_dtype(), shape)
    if isinstance(lse, torch.Tensor):
        _tensor(lse, "lse", torch.float32, (desc.B, desc.H, desc.n))
    if isinstance(score_partials, torch.Tensor):
        _min_bytes(_tensor(score_partials, "score_partials", torch.float32), "score_partials",
                   L.sc_score_partials_size(ctypes.byref(cd)))
    if isinstance(band_probs, torch.Tensor):
        _min_bytes(_tensor(band_probs, "band_probs", torch.float32), "band_probs",
                   L.sc_band_probs_size(ctypes.byref(cd)))
    lse_t = _opt(lse, lambda: torch.empty((desc.B, desc.H, desc.n), dtype=torch.float32, device=dev))
    sp = _opt(score_partials, lambda: torch.empty(L.sc_score_partials_size(ctypes.byref(cd)) // 4,
                                                  dtype=torch.float32, device=dev))
    bp = _opt(band_probs, lambda: torch.empty(L.sc_band_probs_size(ctypes.byref(cd)) // 4, dtype=torch.float32,
                                              device=dev))
    wsb = L.sc_window_attention_workspace_size(ctypes.byref(cd))
    ws = _ws(wsb, dev) if workspace is None else _tensor(workspace, "workspace")
    wsb = wsb if workspace is None else workspace.numel() * workspace.element_size()
    _check(L.sc_window_attention(ctypes.byref(cd), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse_t), _ptr(sp),
                                 _ptr(bp), _ptr(ws), wsb, _stream(stream)), "sc_window_attention")
    return out, lse_t, sp, bp


@_on_stream
def sc_window_attention_noalloc(desc: Desc, q, k, v, out, lse=None, score_partials=None, band_probs=None,
                                stream=None):
    """sc_window_attention with the library's static device workspace: the C call allocates nothing, so every
    output is the caller's tensor (or None for the optional ones).  Returns (out, lse, score_partials,
    band_probs)."""
    import torch
    L = load()
    cd = desc.c()
    shape = (desc.B, desc.n, desc.H, desc.d)
    for t, nm in ((q, "q"), (k, "k"), (v, "v"), (out, "out")):
        _tensor(t, nm, desc.torch_dtype(), shape)
    if lse is not None:
        _tensor(lse, "lse", torch.float32, (desc.B, desc.H, desc.n))
    if score_partials is not None:
        _min_bytes(_tensor(score_partials, "score_partials", torch.float32), "score_partials",
                   L.sc_score_partials_size(ctypes.byref(cd)))
    if band_probs is not None:
        _min_bytes(_tensor(band_probs, "band_probs", torch.float32), "band_probs",
                   L.sc_band_probs_size(ctypes.byref(cd)))
    _check(L.sc_window_attention_noalloc(ctypes.byref(cd), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                         _ptr(score_partials), _ptr(band_probs), _stream(stream)),
           "sc_window_attention_noalloc")
    return out, lse, score_partials, band_probs


def sc_ltp_score_workspace_size(desc: Desc, mode: int = SC_SCORE_FROM_PARTIALS) -> int:
    return load().sc_ltp_score_workspace_size(ctypes.byref(desc.c()), mode)


@_on_stream
def sc_ltp_score(desc: Desc, src, mode: int = SC_SCORE_FROM_PARTIALS, scores=None, workspace=None, stream=None):
    import torch
    L = load()
    cd = desc.c()
    need = L.sc_score_partials_size(ctypes.byref(cd)) if mode == SC_SCORE_FROM_PARTIALS else \
        L.sc_band_probs_size(ctypes.byref(cd))
    _min_bytes(_tensor(src, "src", torch.float32), "src", need)
    scores = torch.empty((desc.B, desc.n), dtype=torch.float32, device=src.device) if scores is None else \
        _tensor(scores, "scores", torch.float32, (desc.B, desc.n))
    wsb = L.sc_ltp_score_workspace_size(ctypes.byref(cd), mode)
    ws = (_ws(wsb, src.device) if wsb > 0 else None) if workspace is None else \
        _min_bytes(_tensor(workspace, "workspace"), "workspace", wsb)
    wsb = wsb if workspace is None else workspace.numel() * workspace.element_size()
    _check(L.sc_ltp_score(ctypes.byref(cd), mode, _ptr(src), _ptr(scores), _ptr(ws), wsb, _stream(stream)),
           "sc_ltp_score")
    return scores


def sc_ltp_prune_compact_workspace_size(desc: Desc) -> int:
    return load().sc_ltp_prune_compact_workspace_size(ctypes.byref(desc.c()))


@_on_stream
def sc_ltp_prune_compact(desc: Desc, scores, threshold, keep_global=True, tensors=(), dsts=None, orig_idx_in=None,
                         want_orig=True, outs=None, workspace=None, stream=None):
    """Threshold rule.  Returns (keep_idx, new_len, new_global_pos, orig_idx_out, dsts).

    outs: optional dict of preallocated keep_idx / new_len / new_global_pos / orig_idx_out."""
    return _prune_compact("sc_ltp_prune_compact", desc, scores, threshold, keep_global, tensors, dsts, orig_idx_in,
                          want_orig, outs, workspace, stream)


@_on_stream
def sc_topk_prune_compact(desc: Desc, scores, keep_ratio, keep_global=True, tensors=(), dsts=None, orig_idx_in=None,
                          want_orig=True, outs=None, workspace=None, stream=None):
    """Top-k rule (keep ceil(keep_ratio * candidates) per sequence); same returns as sc_ltp_prune_compact."""
    return _prune_compact("sc_topk_prune_compact", desc, scores, keep_ratio, keep_global, tensors, dsts, orig_idx_in,
                          want_orig, outs, workspace, stream)


def _prune_compact(fn, desc, scores, value, keep_global, tensors, dsts, orig_idx_in, want_orig, outs, workspace,
                   stream):
    import torch
    L = load()
    cd = desc.c()
    B, n, G = desc.B, desc.n, desc.G
    _tensor(scores, "scores", torch.float32, (B, n))
    dev = scores.device
    outs = outs or {}
    for key, shape in (("keep_idx", (B, n)), ("new_len", (B,)), ("new_global_pos", (B, G)),
                       ("orig_idx_out", (B, n))):
        if outs.get(key) is not None:
            _tensor(outs[key], key, torch.int32, shape)
    if orig_idx_in is not None:
        _tensor(orig_idx_in, "orig_idx_in", torch.int32, (B, n))
    keep_idx = outs.get("keep_idx") if "keep_idx" in outs else torch.empty((B, n), dtype=torch.int32, device=dev)
    new_len = outs.get("new_len") if "new_len" in outs else torch.empty((B,), dtype=torch.int32, device=dev)
    ngp = outs.get("new_global_pos") if "new_global_pos" in outs else (
        torch.empty((B, G), dtype=torch.int32, device=dev) if G > 0 else None)
    orig_out = outs.get("orig_idx_out") if "orig_idx_out" in outs else (
        torch.empty((B, n), dtype=torch.int32, device=dev) if want_orig else None)
    tensors = [_tensor(t, f"tensors[{i}]", leading=(B, n)) for i, t in enumerate(tensors)]
    if dsts is None:
        dsts = [torch.empty_like(t) for t in tensors]
    if len(dsts) != len(tensors):
        raise ValueError("dsts: one destination per source tensor")
    for i, (t, o) in enumerate(zip(tensors, dsts)):
        _tensor(o, f"dsts[{i}]", t.dtype, tuple(t.shape))
    nt = len(tensors)
    src_arr = (ctypes.c_void_p * max(nt, 1))(*[t.data_ptr() for t in tensors])
    dst_arr = (ctypes.c_void_p * max(nt, 1))(*[t.data_ptr() for t in dsts])
    rb_arr = (ctypes.c_int64 * max(nt, 1))(*[t.numel() * t.element_size() // (B * n) for t in tensors])
    wsb = L.sc_ltp_prune_compact_workspace_size(ctypes.byref(cd))
    ws = _ws(wsb, dev) if workspace is None else _tensor(workspace, "workspace")
    wsb = wsb if workspace is None else workspace.numel() * workspace.element_size()
    _check(getattr(L, fn)(ctypes.byref(cd), _ptr(scores), ctypes.c_float(value), int(bool(keep_global)), nt, src_arr,
                          dst_arr, rb_arr, _ptr(keep_idx), _ptr(new_len), _ptr(ngp), _ptr(orig_idx_in),
                          _ptr(orig_out), _ptr(ws), wsb, _stream(stream)), fn)
    return keep_idx, new_len, ngp, orig_out, dsts


@_on_stream
def sc_ltp_soft_mask(desc: Desc, scores, theta, temperature, out, keep_global=True, mask=None, y=None,
                     stream=None):
    """Soft mask of LTP's training phase.  Returns (mask [B, n] float32, y = mask * out)."""
    import torch
    L = load()
    shape = (desc.B, desc.n, desc.H, desc.d)
    _tensor(scores, "scores", torch.float32, (desc.B, desc.n))
    _tensor(out, "out", desc.torch_dtype(), shape)
    mask = torch.empty((desc.B, desc.n), dtype=torch.float32, device=out.device) if mask is None else \
        _tensor(mask, "mask", torch.float32, (desc.B, desc.n))
    y = torch.empty_like(out) if y is None else _tensor(y, "y", desc.torch_dtype(), shape)
    _check(L.sc_ltp_soft_mask(ctypes.byref(desc.c()), _ptr(scores), ctypes.c_float(theta),
                              ctypes.c_float(temperature), int(bool(keep_global)), _ptr(out), _ptr(mask), _ptr(y),
                              _stream(stream)), "sc_ltp_soft_mask")
    return mask, y


def sc_ltp_soft_backward_workspace_size(desc: Desc) -> int:
    return load().sc_ltp_soft_backward_workspace_size(ctypes.byref(desc.c()))


@_on_stream
def sc_ltp_soft_backward(desc: Desc, q, k, v, out, lse, mask, temperature, dy, dmask=None, keep_global=True,
                         grads=None, workspace=None, stream=None):
    """Gradients of the soft-pruned layer.  Returns (dq, dk, dv, dtheta [1] float32 on the device).
    grads: optional (dq, dk, dv, dtheta) output tensors."""
    import torch
    L = load()
    cd = desc.c()
    shape = (desc.B, desc.n, desc.H, desc.d)
    for t, nm in ((q, "q"), (k, "k"), (v, "v"), (out, "out"), (dy, "dy")):
        _tensor(t, nm, desc.torch_dtype(), shape)
    _tensor(lse, "lse", torch.float32, (desc.B, desc.H, desc.n))
    _tensor(mask, "mask", torch.float32, (desc.B, desc.n))
    if dmask is not None:
        _tensor(dmask, "dmask", torch.float32, (desc.B, desc.n))
    if grads is not None:
        for t, nm in zip(grads[:3], ("dq", "dk", "dv")):
            _tensor(t, nm, desc.torch_dtype(), shape)
        _tensor(grads[3], "dtheta", torch.float32, (1,))
    if grads is None:
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                 torch.empty(1, dtype=torch.float32, device=q.device))
    dq, dk, dv, dth = grads
    wsb = L.sc_ltp_soft_backward_workspace_size(ctypes.byref(cd))
    ws = _ws(wsb, q.device) if workspace is None else _tensor(workspace, "workspace")
    wsb = wsb if workspace is None else workspace.numel() * workspace.element_size()
    _check(L.sc_ltp_soft_backward(ctypes.byref(cd), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(mask),
                                  ctypes.c_float(temperature), int(bool(keep_global)), _ptr(dy), _ptr(dmask),
                                  _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dth), _ptr(ws), wsb, _stream(stream)),
           "sc_ltp_soft_backward")
    return dq, dk, dv, dth


def _stack_args(desc, x_in, x_out, wqkv, wo, thresholds):
    import torch
    D = desc.H * desc.d
    _tensor(x_in, "x_in", torch.bfloat16, (desc.B, desc.n, D))
    if x_out is not None:
        _tensor(x_out, "x_out", torch.bfloat16, (desc.B, desc.n, D))
    if len(wo) != len(wqkv) or len(thresholds) != len(wqkv):
        raise ValueError("wqkv, wo and thresholds: one per layer")
    for i in range(len(wqkv)):
        _tensor(wqkv[i], f"wqkv[{i}]", torch.bfloat16, (D, 3 * D))
        _tensor(wo[i], f"wo[{i}]", torch.bfloat16, (D, D))


def sc_encoder_attn_stack_workspace_size(desc: Desc, n_layers: int) -> int:
    return load().sc_encoder_attn_stack_workspace_size(ctypes.byref(desc.c()), int(n_layers))


@_on_stream
def sc_encoder_attn_stack(desc: Desc, x_in, wqkv, wo, thresholds, keep_global=True, ln_eps=1e-5, x_out=None,
                          workspace=None, stream=None):
    """Returns (x_out, final_len, orig_idx, kept_per_layer)."""
    import torch
    L = load()
    cd = desc.c()
    nl = len(wqkv)
    B, n = desc.B, desc.n
    _stack_args(desc, x_in, x_out, wqkv, wo, thresholds)
    dev = x_in.device
    x_out = torch.empty_like(x_in) if x_out is None else x_out
    final_len = torch.empty((B,), dtype=torch.int32, device=dev)
    orig = torch.empty((B, n), dtype=torch.int32, device=dev)
    kpl = torch.empty((nl, B), dtype=torch.int32, device=dev)
    wq = (ctypes.c_void_p * nl)(*[w.data_ptr() for w in wqkv])
    wo_ = (ctypes.c_void_p * nl)(*[w.data_ptr() for w in wo])
    th = (ctypes.c_float * nl)(*[float(t) for t in thresholds])
    wsb = L.sc_encoder_attn_stack_workspace_size(ctypes.byref(cd), nl)
    ws = _ws(wsb, dev) if workspace is None else _min_bytes(_tensor(workspace, "workspace"), "workspace", wsb)
    _check(L.sc_encoder_attn_stack(ctypes.byref(cd), nl, _ptr(x_in), wq, wo_, th, int(bool(keep_global)),
                                   ctypes.c_float(ln_eps), _ptr(x_out), _ptr(final_len), _ptr(orig), _ptr(kpl),
                                   _ptr(ws), wsb, _stream(stream)), "sc_encoder_attn_stack")
    return x_out, final_len, orig, kpl


def sc_encoder_stack_workspace_size(desc: Desc, n_layers: int, ffn_dim: int) -> int:
    return load().sc_encoder_stack_workspace_size(ctypes.byref(desc.c()), int(n_layers), int(ffn_dim))


@_on_stream
def sc_encoder_stack(desc: Desc, x_in, wqkv, wo, w1, w2, thresholds, windows=None, keep_global=True, ln_eps=1e-5,
                     x_out=None, workspace=None, stream=None):
    """Full stack (feed-forward block, per-layer windows).  Returns (x_out, final_len, orig_idx, kept_per_layer)."""
    import torch
    L = load()
    cd = desc.c()
    nl = len(wqkv)
    B, n = desc.B, desc.n
    _stack_args(desc, x_in, x_out, wqkv, wo, thresholds)
    F = int(w1[0].shape[1])
    D = desc.H * desc.d
    if len(w1) != nl or len(w2) != nl or (windows is not None and len(windows) != nl):
        raise ValueError("w1, w2 and windows: one per layer")
    for i in range(nl):
        _tensor(w1[i], f"w1[{i}]", torch.bfloat16, (D, F))
        _tensor(w2[i], f"w2[{i}]", torch.bfloat16, (F, D))
    dev = x_in.device
    x_out = torch.empty_like(x_in) if x_out is None else x_out
    final_len = torch.empty((B,), dtype=torch.int32, device=dev)
    orig = torch.empty((B, n), dtype=torch.int32, device=dev)
    kpl = torch.empty((nl, B), dtype=torch.int32, device=dev)
    arr = lambda ts: (ctypes.c_void_p * nl)(*[t.data_ptr() for t in ts])  # noqa: E731
    th = (ctypes.c_float * nl)(*[float(t) for t in thresholds])
    win = None if windows is None else (ctypes.c_int32 * nl)(*[int(w) for w in windows])
    wsb = L.sc_encoder_stack_workspace_size(ctypes.byref(cd), nl, F)
    ws = _ws(wsb, dev) if workspace is None else _min_bytes(_tensor(workspace, "workspace"), "workspace", wsb)
    _check(L.sc_encoder_stack(ctypes.byref(cd), nl, win, _ptr(x_in), arr(wqkv), arr(wo), arr(w1), arr(w2), F, th,
                              int(bool(keep_global)), ctypes.c_float(ln_eps), _ptr(x_out), _ptr(final_len),
                              _ptr(orig), _ptr(kpl), _ptr(ws), wsb, _stream(stream)), "sc_encoder_stack")
    return x_out, final_len, orig, kpl


@_on_stream
def sc_validate_desc(desc: Desc, err=None, stream=None):
    """Enqueues the check of the descriptor's device arrays (valid_len, global_pos); returns the int32 [1]
    device tensor that receives the OR of the SC_VALID_* bits of the violations found (0: none)."""
    import torch
    L = load()
    cd = desc.c()
    if err is None:
        err = torch.empty(1, dtype=torch.int32, device=desc.valid_len.device)
    _tensor(err, "err", torch.int32, (1,))
    _check(L.sc_validate_desc(ctypes.byref(cd), _ptr(err), _stream(stream)), "sc_validate_desc")
    return err


def sc_profile_window_kernel(enable: bool):
    _check(load().sc_profile_window_kernel(int(bool(enable))), "sc_profile_window_kernel")


def sc_profile_window_kernel_read(capacity: int = 4096):
    """Per window-attention call since the last enable/read, in call order: (launch-1 milliseconds, launch-2
    milliseconds), as two lists."""
    fwd = (ctypes.c_double * capacity)()
    cols = (ctypes.c_double * capacity)()
    cnt = ctypes.c_int64(0)
    _check(load().sc_profile_window_kernel_read(fwd, cols, capacity, ctypes.byref(cnt)),
           "sc_profile_window_kernel_read")
    k = min(cnt.value, capacity)
    return list(fwd[:k]), list(cols[:k])
