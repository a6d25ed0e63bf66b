"""Thin ctypes binding of ``include/ffn_sparse.h`` (argument marshalling only).

Every function takes torch device tensors, checks the dtypes, shapes and devices the
C ABI cannot see (it receives bare pointers and sizes), and passes raw device pointers
plus a HIP stream (by default the current stream of the tensors' device) to the C ABI.  All arithmetic runs in the gfx950 kernels of
``libffn_sparse.so``; there is no fallback: if the library is missing this module
raises on first use.
"""
from __future__ import annotations

import ctypes
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libffn_sparse.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "ffn_sparse.h")
HEADERS = [HEADER, os.path.join(os.path.dirname(PKG), "include", "ffn_lopa_approx.h")]

FFN_F32 = 0
FFN_BF16 = 1
FFN_I8 = 2
FFN_I4 = 3

STATUS = {0: "FFN_OK", -1: "FFN_ERR_NULL", -2: "FFN_ERR_SHAPE", -3: "FFN_ERR_DTYPE", -4: "FFN_ERR_ALIGN",
          -5: "FFN_ERR_WORKSPACE", -6: "FFN_ERR_HIP", -7: "FFN_ERR_OPTION"}

FFN_ACT_RELU = 0
FFN_ACT_RSPLUS = 1


class Scales(ctypes.Structure):
    """``ffn_scales_t``: fp32 row scales of quantized weights (device pointers)."""
    _fields_ = [("gate", ctypes.c_void_p), ("lopa_a", ctypes.c_void_p), ("lopa_b", ctypes.c_void_p),
                ("up", ctypes.c_void_p), ("down", ctypes.c_void_p)]


class Options(ctypes.Structure):
    """``ffn_options_t``: the paper's full FFN form (activation, SiLU on W_up, G, RMSNorm)."""
    _fields_ = [("act", ctypes.c_int), ("silu_up", ctypes.c_int), ("g_idx", ctypes.c_void_p),
                ("g_sign", ctypes.c_void_p), ("rms_norm", ctypes.c_int), ("rms_gain", ctypes.c_void_p),
                ("rms_eps", ctypes.c_float)]


class FFNError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} failed: {STATUS.get(code, code)}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_31975_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i, f, vp, sz = ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
        L.ffn_workspace_bytes.restype = sz
        L.ffn_workspace_bytes.argtypes = [i, i, i, i]
        std = [i, i, i, i, vp, vp, vp, vp, f, vp, vp, sz, vp]
        lop = [i, i, i, i, i, vp, vp, vp, vp, vp, f, vp, vp, sz, vp]
        op = ctypes.POINTER(Options)
        sp = ctypes.POINTER(Scales)
        std_ex = std[:9] + [op] + std[9:]
        lop_ex = lop[:11] + [op] + lop[11:]
        std_q = std[:8] + [sp] + std[8:9] + [op] + std[9:]
        lop_q = lop[:10] + [sp] + lop[10:11] + [op] + lop[11:]
        for name, args in (("ffn_dense_forward", std), ("ffn_sparse_forward", std),
                           ("ffn_lopa_sparse_forward", lop), ("ffn_lopa_dense_forward", lop),
                           ("ffn_dense_forward_ex", std_ex), ("ffn_sparse_forward_ex", std_ex),
                           ("ffn_lopa_sparse_forward_ex", lop_ex), ("ffn_lopa_dense_forward_ex", lop_ex),
                           ("ffn_dense_forward_q", std_q), ("ffn_sparse_forward_q", std_q),
                           ("ffn_lopa_sparse_forward_q", lop_q), ("ffn_lopa_dense_forward_q", lop_q)):
            getattr(L, name).restype = i
            getattr(L, name).argtypes = args
        L.ffn_active_set.restype = i
        L.ffn_active_set.argtypes = [vp, i, i, i, i, vp, vp, vp, vp]
        L.ffn_sparse_forward_noalloc.restype = i
        L.ffn_sparse_forward_noalloc.argtypes = [i, i, i, i, vp, vp, vp, vp, f, vp, vp]
        pp = ctypes.POINTER(ctypes.c_void_p)
        L.ffn_workspace_active.restype = i
        L.ffn_workspace_active.argtypes = [vp, i, i, i, i, pp, pp, pp, pp]
        L.ffn_time_next_gate_kernel.restype = i
        L.ffn_time_next_gate_kernel.argtypes = [vp, vp]
        L.ffn_set_z_wait_ticks.restype = i
        L.ffn_set_z_wait_ticks.argtypes = [ctypes.c_uint64]
        L.ffn_lopa_approx_workspace_bytes.restype = sz
        L.ffn_lopa_approx_workspace_bytes.argtypes = [i, i, i]
        L.ffn_lopa_approx.restype = i
        L.ffn_lopa_approx.argtypes = [i, i, i, vp, i, vp, vp, vp, vp, ctypes.POINTER(ctypes.c_int),
                                      ctypes.POINTER(ctypes.c_double), vp, sz, vp]
        L.ffn_status_string.restype = ctypes.c_char_p
        L.ffn_status_string.argtypes = [i]
        _lib = L
    return _lib


def declared_functions() -> list[str]:
    """Names of the functions the public headers declare."""
    text = "".join(open(h).read() for h in HEADERS)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+[\s*]+(ffn_\w+)\s*\(", text, re.M)))


# ---------------------------------------------------------------- marshalling helpers
def _torch():
    import torch
    return torch


def weight_dtype(w) -> int:
    torch = _torch()
    if w.dtype == torch.bfloat16:
        return FFN_BF16
    if w.dtype == torch.float32:
        return FFN_F32
    raise TypeError(f"weights must be bfloat16 or float32, got {w.dtype}")


def quant_dtype(w, d: int) -> int:
    """FFN_I8 for int8 codes of row length d, FFN_I4 for uint8 bytes holding d/2 code pairs."""
    torch = _torch()
    if w.dtype == torch.int8 and w.shape[-1] == d:
        return FFN_I8
    if w.dtype == torch.uint8 and 2 * w.shape[-1] == d:
        return FFN_I4
    raise TypeError(f"quantized weights must be int8 [.., d] or uint8 [.., d/2], got {w.dtype} {tuple(w.shape)}")


def scales(gate=None, lopa_a=None, lopa_b=None, up=None, down=None) -> Scales:
    """Build an ``ffn_scales_t`` from float32 device tensors (or None)."""
    return Scales(*(_dev(t, n) for t, n in ((gate, "gate"), (lopa_a, "lopa_a"), (lopa_b, "lopa_b"), (up, "up"),
                                             (down, "down"))))


def _dev(t, what):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous device tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    """The HIP stream to enqueue on: `stream`, or the current stream of the tensors' device
    (not of the current device, which may be another one)."""
    torch = _torch()
    s = torch.cuda.current_stream(device) if stream is None else stream
    if s.device != device:
        raise ValueError(f"stream is on {s.device}, the tensors on {device}")
    return ctypes.c_void_p(s.cuda_stream)


def _check(fn, rc):
    if rc != 0:
        raise FFNError(fn, rc)


def workspace_bytes(T: int, d: int, d_ff: int, r: int = 0) -> int:
    return int(lib().ffn_workspace_bytes(T, d, d_ff, r))


def alloc_workspace(T: int, d: int, d_ff: int, r: int = 0, device="cuda"):
    """A zero-filled workspace (the header asks for zeros before the first call)."""
    torch = _torch()
    n = workspace_bytes(T, d, d_ff, r)
    if n == 0:
        raise FFNError("ffn_workspace_bytes", -2)
    return torch.zeros(n, dtype=torch.uint8, device=device)


def options(act=FFN_ACT_RELU, silu_up=False, g_idx=None, g_sign=None, rms_norm=False, rms_gain=None,
            rms_eps=0.0) -> Options:
    """Build an ``ffn_options_t``; g_idx (int32), g_sign (int8) and rms_gain (float32) are
    device tensors or None.  The tensors must outlive the call's work on its stream."""
    return Options(int(act), 1 if silu_up else 0, _dev(g_idx, "g_idx"), _dev(g_sign, "g_sign"),
                   1 if rms_norm else 0, _dev(rms_gain, "rms_gain"), float(rms_eps))


def _opt(opt):
    return None if opt is None else ctypes.byref(opt)


def _check_args(x, y, ws, weights, cols_of):
    """Validate what the C ABI cannot see: x and y are float32 [T, d] on one device, every
    weight has w_up's dtype and its expected [rows, cols] shape (``weights`` maps a name to
    (tensor, rows, logical cols)), and the workspace is on the same device.  cols_of(n)
    gives the stored row length of n logical elements (n / 2 bytes for int4 codes)."""
    torch = _torch()
    if x.dim() != 2 or x.dtype != torch.float32:
        raise ValueError(f"x must be a float32 [T, d] tensor, got {x.dtype} {tuple(x.shape)}")
    if y.dtype != torch.float32 or tuple(y.shape) != tuple(x.shape):
        raise ValueError(f"y must be float32 of x's shape {tuple(x.shape)}, got {y.dtype} {tuple(y.shape)}")
    dev = x.device
    if y.device != dev or ws.device != dev:
        raise ValueError("x, y and the workspace must be on one device")
    wdtype = weights["w_up"][0].dtype
    for name, (w, rows, cols) in weights.items():
        if w is None:
            raise ValueError(f"{name} is required")
        if w.dtype != wdtype:
            raise ValueError(f"{name} is {w.dtype}, w_up is {wdtype}: every weight must have one dtype")
        if w.device != dev:
            raise ValueError(f"{name} must be on x's device")
        if tuple(w.shape) != (rows, cols_of(cols)):
            raise ValueError(f"{name} must be [{rows}, {cols_of(cols)}], got {tuple(w.shape)}")


def _same(n):
    return n


def _std_call(name, x, w_gate, w_up, w_down_t, t, y, ws, stream, opt=()):
    T, d = x.shape
    d_ff = w_up.shape[0]
    _check_args(x, y, ws, {"w_up": (w_up, d_ff, d), "w_gate": (w_gate, d_ff, d), "w_down_t": (w_down_t, d_ff, d)},
                _same)
    rc = getattr(lib(), name)(weight_dtype(w_up), T, d, d_ff, _dev(x, "x"), _dev(w_gate, "w_gate"),
                              _dev(w_up, "w_up"), _dev(w_down_t, "w_down_t"), ctypes.c_float(t), *opt,
                              _dev(y, "y"), _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream, x.device))
    _check(name, rc)
    return y


def _lopa_call(name, x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream, opt=()):
    T, d = x.shape
    d_ff, r = lopa_b.shape
    _check_args(x, y, ws, {"w_up": (w_up, d_ff, d), "lopa_a": (lopa_a, r, d), "lopa_b": (lopa_b, d_ff, r),
                           "w_down_t": (w_down_t, d_ff, d)}, _same)
    rc = getattr(lib(), name)(weight_dtype(w_up), T, d, d_ff, r, _dev(x, "x"), _dev(lopa_a, "lopa_a"),
                              _dev(lopa_b, "lopa_b"), _dev(w_up, "w_up"), _dev(w_down_t, "w_down_t"),
                              ctypes.c_float(t), *opt, _dev(y, "y"), _dev(ws, "ws"),
                              ws.numel() * ws.element_size(), _stream(stream, x.device))
    _check(name, rc)
    return y


# ---------------------------------------------------------------- the C ABI, by name
def ffn_dense_forward(x, w_gate, w_up, w_down_t, t, y, ws, stream=None):
    return _std_call("ffn_dense_forward", x, w_gate, w_up, w_down_t, t, y, ws, stream)


def ffn_sparse_forward(x, w_gate, w_up, w_down_t, t, y, ws, stream=None):
    return _std_call("ffn_sparse_forward", x, w_gate, w_up, w_down_t, t, y, ws, stream)


def ffn_sparse_forward_noalloc(x, w_gate, w_up, w_down_t, t, y, stream=None):
    """ffn_sparse_forward with the library's own per-GPU workspace (no allocation; calls that
    overlap on one GPU race)."""
    T, d = x.shape
    d_ff = w_up.shape[0]
    _check_args(x, y, y, {"w_up": (w_up, d_ff, d), "w_gate": (w_gate, d_ff, d), "w_down_t": (w_down_t, d_ff, d)},
                _same)
    rc = lib().ffn_sparse_forward_noalloc(weight_dtype(w_up), T, d, d_ff, _dev(x, "x"), _dev(w_gate, "w_gate"),
                                          _dev(w_up, "w_up"), _dev(w_down_t, "w_down_t"), ctypes.c_float(t),
                                          _dev(y, "y"), _stream(stream, x.device))
    _check("ffn_sparse_forward_noalloc", rc)
    return y


def ffn_lopa_sparse_forward(x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream=None):
    return _lopa_call("ffn_lopa_sparse_forward", x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream)


def ffn_lopa_dense_forward(x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream=None):
    return _lopa_call("ffn_lopa_dense_forward", x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream)


def ffn_dense_forward_ex(x, w_gate, w_up, w_down_t, t, opt, y, ws, stream=None):
    return _std_call("ffn_dense_forward_ex", x, w_gate, w_up, w_down_t, t, y, ws, stream, (_opt(opt),))


def ffn_sparse_forward_ex(x, w_gate, w_up, w_down_t, t, opt, y, ws, stream=None):
    return _std_call("ffn_sparse_forward_ex", x, w_gate, w_up, w_down_t, t, y, ws, stream, (_opt(opt),))


def ffn_lopa_sparse_forward_ex(x, lopa_a, lopa_b, w_up, w_down_t, t, opt, y, ws, stream=None):
    return _lopa_call("ffn_lopa_sparse_forward_ex", x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream,
                      (_opt(opt),))


def ffn_lopa_dense_forward_ex(x, lopa_a, lopa_b, w_up, w_down_t, t, opt, y, ws, stream=None):
    return _lopa_call("ffn_lopa_dense_forward_ex", x, lopa_a, lopa_b, w_up, w_down_t, t, y, ws, stream,
                      (_opt(opt),))


def _q_call(name, x, gate, lopa_a, w_up, w_down_t, sc, t, opt, y, ws, stream, r):
    T, d = x.shape
    d_ff = w_up.shape[0]
    wdt = quant_dtype(w_up, d) if w_up.dtype != _torch().float32 and w_up.dtype != _torch().bfloat16 \
        else weight_dtype(w_up)
    cols_of = (lambda n: n // 2) if wdt == FFN_I4 else _same
    if wdt == FFN_I4 and (d % 2 or r % 2):
        raise ValueError("int4 codes need an even d (and r)")
    ws_ = {"w_up": (w_up, d_ff, d), "w_down_t": (w_down_t, d_ff, d)}
    if r:
        ws_.update(lopa_a=(lopa_a, r, d), lopa_b=(gate, d_ff, r))
    else:
        ws_.update(w_gate=(gate, d_ff, d))
    _check_args(x, y, ws, ws_, cols_of)
    head = [wdt, T, d, d_ff] + ([r] if r else [])
    ptrs = [_dev(x, "x")] + ([_dev(lopa_a, "lopa_a")] if r else []) + [_dev(gate, "gate"), _dev(w_up, "w_up"),
                                                                       _dev(w_down_t, "w_down_t")]
    rc = getattr(lib(), name)(*head, *ptrs, None if sc is None else ctypes.byref(sc), ctypes.c_float(t), _opt(opt),
                              _dev(y, "y"), _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream, x.device))
    _check(name, rc)
    return y


def ffn_dense_forward_q(x, w_gate, w_up, w_down_t, sc, t, opt, y, ws, stream=None):
    return _q_call("ffn_dense_forward_q", x, w_gate, None, w_up, w_down_t, sc, t, opt, y, ws, stream, 0)


def ffn_sparse_forward_q(x, w_gate, w_up, w_down_t, sc, t, opt, y, ws, stream=None):
    return _q_call("ffn_sparse_forward_q", x, w_gate, None, w_up, w_down_t, sc, t, opt, y, ws, stream, 0)


def ffn_lopa_sparse_forward_q(x, lopa_a, lopa_b, w_up, w_down_t, sc, t, opt, y, ws, stream=None):
    r = lopa_a.shape[0]
    return _q_call("ffn_lopa_sparse_forward_q", x, lopa_b, lopa_a, w_up, w_down_t, sc, t, opt, y, ws, stream, r)


def ffn_lopa_dense_forward_q(x, lopa_a, lopa_b, w_up, w_down_t, sc, t, opt, y, ws, stream=None):
    r = lopa_a.shape[0]
    return _q_call("ffn_lopa_dense_forward_q", x, lopa_b, lopa_a, w_up, w_down_t, sc, t, opt, y, ws, stream, r)


def ffn_active_set(ws, T, d, d_ff, r=0, stream=None, with_act=True):
    """Returns (idx [n] int32 numpy, act [T, n] float32 numpy or None) of the last call."""
    import numpy as np
    n = ctypes.c_int32(0)
    idx = np.empty(d_ff, np.int32)
    act = np.empty((T, d_ff), np.float32) if with_act else None
    rc = lib().ffn_active_set(_dev(ws, "ws"), T, d, d_ff, r, ctypes.byref(n), idx.ctypes.data_as(ctypes.c_void_p),
                              None if act is None else act.ctypes.data_as(ctypes.c_void_p),
                              _stream(stream, ws.device))
    _check("ffn_active_set", rc)
    k = n.value
    return idx[:k].copy(), (None if act is None else act[:, :k].copy())


def ffn_workspace_active(ws, T, d, d_ff, r=0):
    """Device views of the last call's active set (no synchronization, nothing enqueued):
    returns (meta, seg_count, idx, act) as tensors aliasing the workspace ``ws``: meta int32
    [64] (meta[0] = nseg), seg_count int32 [d_ff] (the first nseg entries are the segment
    counts), idx int32 [d_ff], act float32 [T, d_ff]."""
    torch = _torch()
    if ws.dtype != torch.uint8 or not ws.is_contiguous():
        raise ValueError("ws must be a contiguous uint8 tensor")
    ptrs = [ctypes.c_void_p() for _ in range(4)]
    rc = lib().ffn_workspace_active(_dev(ws, "ws"), T, d, d_ff, r, *(ctypes.byref(p) for p in ptrs))
    _check("ffn_workspace_active", rc)
    base = ws.data_ptr()
    views = []
    for p, n, dt in zip(ptrs, (64, d_ff, d_ff, T * d_ff), (torch.int32, torch.int32, torch.int32, torch.float32)):
        off = p.value - base
        nbytes = 4 * n
        if off < 0 or off + nbytes > ws.numel():
            raise FFNError("ffn_workspace_active", -5)
        views.append(ws[off:off + nbytes].view(dt))
    return views[0], views[1], views[2], views[3].view(T, d_ff)


def ffn_time_next_gate_kernel(start, stop):
    """Arm torch.cuda.Event pair (enable_timing=True) for the next call's gate kernel."""
    rc = lib().ffn_time_next_gate_kernel(ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event))
    _check("ffn_time_next_gate_kernel", rc)


def ffn_set_z_wait_ticks(ticks: int):
    """Set the single-token LoPA gate kernel's bounded wait for z (100 MHz ticks; test hook)."""
    _check("ffn_set_z_wait_ticks", lib().ffn_set_z_wait_ticks(int(ticks)))


Z_WAIT_TICKS_DEFAULT = 10000  # 100 us, the library's default


def ffn_lopa_approx(w, r: int, max_iters: int = 20, stream=None):
    """LoPA approximation of a gate matrix w ([H, D] float32 device tensor): returns
    (g_idx int32 [H], g_sign int8 [H], lopa_b = U [H, r] f32, lopa_a = V [r, D] f32,
    iters, objective), the arrays as device tensors."""
    torch = _torch()
    H, D = w.shape
    n = int(lib().ffn_lopa_approx_workspace_bytes(H, D, r))
    if n == 0:
        raise FFNError("ffn_lopa_approx_workspace_bytes", -2)
    ws = torch.empty(n, dtype=torch.uint8, device=w.device)
    g_idx = torch.empty(H, dtype=torch.int32, device=w.device)
    g_sign = torch.empty(H, dtype=torch.int8, device=w.device)
    U = torch.empty((H, r), dtype=torch.float32, device=w.device)
    V = torch.empty((r, D), dtype=torch.float32, device=w.device)
    it, obj = ctypes.c_int(0), ctypes.c_double(0.0)
    rc = lib().ffn_lopa_approx(H, D, r, _dev(w, "w"), max_iters, _dev(g_idx, "g_idx"), _dev(g_sign, "g_sign"),
                               _dev(U, "lopa_b"), _dev(V, "lopa_a"), ctypes.byref(it), ctypes.byref(obj),
                               _dev(ws, "ws"), n, _stream(stream, w.device))
    _check("ffn_lopa_approx", rc)
    return g_idx, g_sign, U, V, it.value, obj.value


def ffn_status_string(code: int) -> str:
    return lib().ffn_status_string(code).decode()
