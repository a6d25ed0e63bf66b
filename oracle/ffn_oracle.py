"""Python front end of the reference oracle (test infrastructure, not product).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  It builds ``ffn_oracle.c`` with gcc into
``oracle/_build/`` and calls it through ctypes.  Nothing here is shared with the
GPU library: no headers, no helpers, no constants.

The computation (gated FFN of Section 3.1, Eq. (ffn); shifted-ReLU or shifted R-S+
activation; skipping of inactive neurons per Section 3.1 "FFN FLOP-ratio"; LoPA gate
h = G x + U (V x), optionally with RMSNorm between the factors, Section 3.3,
Eq. (lopaapprox); the double activation of Section 3.3) is documented in
``ffn_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ffn_oracle.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD, "libffn_oracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, no FMA contraction)."""
    os.makedirs(_BUILD, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math",
                               "-Wall", "-Wextra", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        vp = ctypes.c_void_p
        i, f = ctypes.c_int, ctypes.c_float
        lib.oracle_ffn_q.restype = i
        lib.oracle_ffn_q.argtypes = [i, i, i, i, i, i, i, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, f, i, i, vp, vp,
                                     i, vp, f, vp, vp, vp, vp, vp]
        _lib = lib
    return _lib


@dataclass
class OracleResult:
    h: np.ndarray        # [T, d_ff] fp64 gate pre-activations
    active: np.ndarray   # [T, d_ff] bool, h > t
    y: np.ndarray        # [T, d] fp64
    macs: np.ndarray     # [T] int64 multiply-adds executed
    z: np.ndarray | None  # [T, r] fp64 (LoPA only)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


_WDTYPE = {0: np.float32, 1: np.uint16, 2: np.int8, 3: np.uint8}


def _weights(w, wdt):
    if w is None:
        return None
    want = _WDTYPE[wdt]
    w = np.ascontiguousarray(w)
    if w.dtype != want:
        raise TypeError(f"weights must be {want.__name__} for wdt={wdt}, got {w.dtype}")
    return w


def _cols(w, wdt):
    """Logical row length of a stored matrix (int4 packs two codes a byte)."""
    return w.shape[1] * (2 if wdt == 3 else 1)


def ffn(x, *, w_up, w_down_t, t, wdt, w_gate=None, lopa_a=None, lopa_b=None,
        skip_inactive=True, act=0, silu_up=False, g_idx=None, g_sign=None, rms_norm=False,
        rms_gain=None, rms_eps=1e-6, scales=None) -> OracleResult:
    """Run the oracle on every token of ``x`` ([T, d] float32).

    Weights: float32 arrays (wdt=0), uint16 arrays holding bfloat16 bit patterns
    (wdt=1), int8 codes (wdt=2) or uint8 arrays of two int4 codes a byte, element 2k in
    the low nibble (wdt=3), row-major: w_gate/w_up/w_down_t [d_ff, d], lopa_a [r, d],
    lopa_b [d_ff, r] (int4: half the columns).  Quantized weights take ``scales``, a dict
    of float32 row scales: gate [d_ff] or a [r] and b [d_ff], up [d_ff], down [d_ff].
    Exactly one of ``w_gate`` (standard gating) or ``lopa_a``+``lopa_b`` (LoPA) is given.
    ``skip_inactive`` selects the sparse method (True) or the dense FFN (False).
    ``act``: 0 shifted ReLU, 1 shifted R-S+; ``silu_up``: SiLU on the W3 output.
    LoPA only: ``g_idx`` (int32 [d_ff]) and ``g_sign`` (int8 [d_ff], +1/-1) give the
    fixed term G; ``rms_norm`` puts RMSNorm (gain ``rms_gain`` [r] or ones, ``rms_eps``)
    between A and B.
    """
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    T, d = x.shape
    w_up = _weights(w_up, wdt)
    w_down_t = _weights(w_down_t, wdt)
    d_ff = w_up.shape[0]
    lopa = lopa_a is not None
    if lopa == (w_gate is not None):
        raise ValueError("give exactly one of w_gate or (lopa_a, lopa_b)")
    w_gate = _weights(w_gate, wdt)
    lopa_a = _weights(lopa_a, wdt)
    lopa_b = _weights(lopa_b, wdt)
    r = lopa_a.shape[0] if lopa else 0
    if w_up.shape[0] != d_ff or _cols(w_up, wdt) != d or w_down_t.shape[0] != d_ff or _cols(w_down_t, wdt) != d:
        raise ValueError("w_up and w_down_t must be [d_ff, d]")
    if not lopa and (w_gate.shape[0] != d_ff or _cols(w_gate, wdt) != d):
        raise ValueError("w_gate must be [d_ff, d]")
    if lopa and (lopa_a.shape[0] != r or _cols(lopa_a, wdt) != d or lopa_b.shape[0] != d_ff or
                 _cols(lopa_b, wdt) != r):
        raise ValueError("lopa_a must be [r, d] and lopa_b [d_ff, r]")
    sc = {}
    if wdt >= 2:
        if scales is None:
            raise ValueError("quantized weights need row scales")
        want = dict(up=d_ff, down=d_ff, **(dict(a=r, b=d_ff) if lopa else dict(gate=d_ff)))
        for k, n in want.items():
            v = np.ascontiguousarray(scales[k], dtype=np.float32)
            if v.shape != (n,):
                raise ValueError(f"scales[{k!r}] must be [{n}]")
            sc[k] = v

    h = np.empty((T, d_ff), np.float64)
    active = np.empty((T, d_ff), np.uint8)
    y = np.empty((T, d), np.float64)
    macs = np.empty((T,), np.int64)
    z = np.empty((T, r), np.float64) if lopa else None
    gi = None if g_idx is None else np.ascontiguousarray(g_idx, dtype=np.int32)
    gs = None if g_sign is None else np.ascontiguousarray(g_sign, dtype=np.int8)
    gain = None if rms_gain is None else np.ascontiguousarray(rms_gain, dtype=np.float32)
    if (gi is not None and gi.shape != (d_ff,)) or (gs is not None and gs.shape != (d_ff,)):
        raise ValueError("g_idx and g_sign must be [d_ff]")
    if gain is not None and gain.shape != (r,):
        raise ValueError("rms_gain must be [r]")
    rc = lib.oracle_ffn_q(1 if lopa else 0, 1 if skip_inactive else 0, wdt, T, d, d_ff, r,
                          _ptr(x), _ptr(w_gate), _ptr(lopa_a), _ptr(lopa_b), _ptr(w_up), _ptr(w_down_t),
                          _ptr(sc.get("gate")), _ptr(sc.get("a")), _ptr(sc.get("b")), _ptr(sc.get("up")),
                          _ptr(sc.get("down")), ctypes.c_float(np.float32(t)), int(act), 1 if silu_up else 0,
                          _ptr(gi), _ptr(gs), 1 if rms_norm else 0, _ptr(gain), ctypes.c_float(np.float32(rms_eps)),
                          _ptr(h), _ptr(z), _ptr(active), _ptr(y), _ptr(macs))
    if rc != 0:
        raise ValueError(f"oracle_ffn_q rejected its arguments (rc={rc})")
    return OracleResult(h=h, active=active.astype(bool), y=y, macs=macs, z=z)
