"""The C ABI library: loads, exports what the header declares, and rejects bad
arguments on the host before anything is enqueued (CPU only: every call here fails
validation, so no kernel is ever launched)."""
import ctypes

import pytest

from paper_2609_31975_amd import ffn

L = None


def setup_module(_):
    global L
    L = ffn.lib()


def test_exports_every_declared_function():
    names = ffn.declared_functions()
    assert set(names) >= {"ffn_workspace_bytes", "ffn_dense_forward", "ffn_sparse_forward",
                          "ffn_lopa_sparse_forward", "ffn_lopa_dense_forward", "ffn_active_set",
                          "ffn_status_string", "ffn_time_next_gate_kernel"}
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    for code, name in ffn.STATUS.items():
        assert ffn.ffn_status_string(code) and ffn.ffn_status_string(code) != "unknown status", name
    assert ffn.ffn_status_string(123) == "unknown status"


def test_workspace_bytes():
    a = ffn.workspace_bytes(1, 4096, 14336, 0)
    b = ffn.workspace_bytes(1, 4096, 14336, 512)
    c = ffn.workspace_bytes(8, 4096, 14336, 512)
    assert 0 < a <= b < c
    assert a % 256 == 0
    assert ffn.workspace_bytes(2, 4096, 14336, 512) < c < ffn.workspace_bytes(9, 4096, 14336, 512)
    # per-token state grows linearly with tokens up to the 64-token pass size, then stops
    assert ffn.workspace_bytes(64, 64, 100, 0) == ffn.workspace_bytes(500, 64, 100, 0)
    for bad in [(0, 8, 8, 0), (1, 0, 8, 0), (1, 8, 0, 0), (1, 8, 8, -1), (1, 1 << 20, 1 << 12, 0)]:
        assert ffn.workspace_bytes(*bad) == 0, bad


A = 1 << 20                     # a 16-byte-aligned address that is never dereferenced
MIS = A + 4                     # misaligned


def _std(fn="ffn_sparse_forward", wdt=1, T=1, d=64, d_ff=128, x=A, g=A, u=A, dn=A, y=A, ws=A, ws_bytes=1 << 30):
    return getattr(L, fn)(wdt, T, d, d_ff, x, g, u, dn, ctypes.c_float(0.5), y, ws, ws_bytes, None)


def _lopa(fn="ffn_lopa_sparse_forward", wdt=1, T=1, d=64, d_ff=128, r=8, x=A, a=A, b=A, u=A, dn=A, y=A, ws=A,
          ws_bytes=1 << 30):
    return getattr(L, fn)(wdt, T, d, d_ff, r, x, a, b, u, dn, ctypes.c_float(0.5), y, ws, ws_bytes, None)


@pytest.mark.parametrize("fn", ["ffn_sparse_forward", "ffn_dense_forward"])
def test_standard_argument_errors(fn):
    assert _std(fn, x=None) == -1
    assert _std(fn, g=None) == -1
    assert _std(fn, dn=None) == -1
    assert _std(fn, y=None) == -1
    assert _std(fn, ws=None) == -1
    assert _std(fn, wdt=7) == -3
    assert _std(fn, T=0) == -2
    assert _std(fn, d=-1) == -2
    assert _std(fn, d_ff=0) == -2
    assert _std(fn, d=1 << 16, d_ff=1 << 15) == -2
    assert _std(fn, x=MIS) == -4
    assert _std(fn, u=MIS) == -4
    assert _std(fn, ws=MIS) == -4
    assert _std(fn, ws_bytes=ffn.workspace_bytes(1, 64, 128, 0) - 1) == -5


@pytest.mark.parametrize("fn", ["ffn_lopa_sparse_forward", "ffn_lopa_dense_forward"])
def test_lopa_argument_errors(fn):
    assert _lopa(fn, a=None) == -1
    assert _lopa(fn, b=None) == -1
    assert _lopa(fn, r=0) == -2
    assert _lopa(fn, wdt=-1) == -3
    assert _lopa(fn, a=MIS) == -4
    assert _lopa(fn, b=MIS) == -4
    assert _lopa(fn, ws_bytes=ffn.workspace_bytes(1, 64, 128, 8) - 256) == -5


def _opt(**kw):
    return ctypes.byref(ffn.Options(**kw))


def _std_ex(opt, fn="ffn_sparse_forward_ex", ws_bytes=1 << 30):
    return getattr(L, fn)(1, 1, 64, 128, A, A, A, A, ctypes.c_float(0.5), opt, A, A, ws_bytes, None)


def _lopa_ex(opt, fn="ffn_lopa_sparse_forward_ex", ws_bytes=1 << 30):
    return getattr(L, fn)(1, 1, 64, 128, 8, A, A, A, A, A, ctypes.c_float(0.5), opt, A, A, ws_bytes, None)


@pytest.mark.parametrize("kind", ["sparse", "dense"])
def test_option_errors(kind):
    std = "ffn_sparse_forward_ex" if kind == "sparse" else "ffn_dense_forward_ex"
    lop = "ffn_lopa_sparse_forward_ex" if kind == "sparse" else "ffn_lopa_dense_forward_ex"
    small = ffn.workspace_bytes(1, 64, 128, 8) - 256
    # a valid option set reaches the workspace check (no launch: the workspace is short)
    assert _lopa_ex(_opt(act=1, silu_up=1, g_idx=A, g_sign=A, rms_norm=1, rms_gain=A, rms_eps=1e-6), lop,
                    small) == -5
    assert _lopa_ex(None, lop, small) == -5
    assert _std_ex(_opt(act=1, silu_up=1), std, ffn.workspace_bytes(1, 64, 128, 0) - 1) == -5
    # invalid option values
    assert _std_ex(_opt(act=2), std) == -7
    assert _std_ex(_opt(act=-1), std) == -7
    assert _std_ex(_opt(silu_up=2), std) == -7
    assert _lopa_ex(_opt(rms_norm=2, rms_eps=1e-6), lop) == -7
    assert _lopa_ex(_opt(g_idx=A), lop) == -7                       # g_sign missing
    assert _lopa_ex(_opt(g_sign=A), lop) == -7                      # g_idx missing
    assert _std_ex(_opt(g_idx=A, g_sign=A), std) == -7              # G belongs to LoPA
    assert _std_ex(_opt(rms_norm=1, rms_eps=1e-6), std) == -7       # so does the norm
    assert _lopa_ex(_opt(rms_norm=1, rms_eps=0.0), lop) == -7
    assert _lopa_ex(_opt(rms_norm=1, rms_eps=-1.0), lop) == -7
    assert _lopa_ex(_opt(rms_norm=1, rms_eps=float("nan")), lop) == -7
    assert _lopa_ex(_opt(rms_norm=1, rms_eps=float("inf")), lop) == -7
    assert _lopa_ex(_opt(rms_gain=A), lop) == -7                    # gain without the norm
    # alignment of the option arrays
    assert _lopa_ex(_opt(g_idx=A + 2, g_sign=A + 1), lop) == -4
    assert _lopa_ex(_opt(rms_norm=1, rms_gain=A + 1, rms_eps=1e-6), lop) == -4


def _q(fn, wdt, sc, d=64, r=0, ws_bytes=1 << 30, T=1):
    if r:
        return getattr(L, fn)(wdt, T, d, 128, r, A, A, A, A, A, sc, ctypes.c_float(0.5), None, A, A, ws_bytes, None)
    return getattr(L, fn)(wdt, T, d, 128, A, A, A, A, sc, ctypes.c_float(0.5), None, A, A, ws_bytes, None)


@pytest.mark.parametrize("kind", ["sparse", "dense"])
def test_quantized_argument_errors(kind):
    std, lop = f"ffn_{kind}_forward_q", f"ffn_lopa_{kind}_forward_q"
    full = ctypes.byref(ffn.Scales(A, A, A, A, A))
    small = ffn.workspace_bytes(1, 64, 128, 0) - 1
    # valid quantized calls reach the workspace check (no launch: the workspace is short)
    for wdt in (ffn.FFN_I8, ffn.FFN_I4):
        assert _q(std, wdt, full, ws_bytes=small) == -5
        assert _q(lop, wdt, full, r=8, ws_bytes=ffn.workspace_bytes(1, 64, 128, 8) - 256) == -5
    assert _q(std, ffn.FFN_BF16, None, ws_bytes=small) == -5      # float weights, no scales
    # the plain and _ex calls take no quantized weights
    assert _std(fn="ffn_sparse_forward", wdt=ffn.FFN_I8) == -3
    assert _lopa(fn="ffn_lopa_sparse_forward", wdt=ffn.FFN_I4) == -3
    assert _q(std, 4, full) == -3
    # scales: required, complete, aligned; none for float weights
    assert _q(std, ffn.FFN_I8, None) == -1
    assert _q(std, ffn.FFN_I8, ctypes.byref(ffn.Scales(None, A, A, A, A))) == -1      # gate missing
    assert _q(std, ffn.FFN_I8, ctypes.byref(ffn.Scales(A, None, None, None, A))) == -1  # up missing
    assert _q(lop, ffn.FFN_I8, ctypes.byref(ffn.Scales(A, None, A, A, A)), r=8) == -1   # A's missing
    assert _q(lop, ffn.FFN_I8, ctypes.byref(ffn.Scales(None, A, A, A, A)), r=8,
              ws_bytes=ffn.workspace_bytes(1, 64, 128, 8) - 256) == -5                 # gate's unused
    assert _q(std, ffn.FFN_I8, ctypes.byref(ffn.Scales(A, None, None, A + 2, A))) == -4
    assert _q(std, ffn.FFN_F32, full) == -7
    # int4 rows must hold whole bytes
    assert _q(std, ffn.FFN_I4, full, d=65) == -2
    assert _q(lop, ffn.FFN_I4, full, r=9) == -2
    assert _q(lop, ffn.FFN_I8, full, r=9, ws_bytes=ffn.workspace_bytes(1, 64, 128, 9) - 256) == -5


def test_lopa_approx_argument_errors():
    n = ffn.workspace_bytes  # noqa: F841 (the forward workspace is unrelated)
    assert L.ffn_lopa_approx_workspace_bytes(0, 8, 1) == 0
    assert L.ffn_lopa_approx_workspace_bytes(8, 8, 9) == 0
    assert L.ffn_lopa_approx_workspace_bytes(1 << 16, 1 << 16, 4) == 0
    ws = L.ffn_lopa_approx_workspace_bytes(64, 32, 4)
    assert ws > 0
    it, obj = ctypes.c_int(), ctypes.c_double()

    def call(H=64, D=32, r=4, w=A, iters=3, ws_bytes=ws, gs=A, it_p=ctypes.byref(it)):
        return L.ffn_lopa_approx(H, D, r, w, iters, A, gs, A, A, it_p, ctypes.byref(obj), A, ws_bytes, None)
    assert call(w=None) == -1
    assert call(it_p=None) == -1
    assert call(r=0) == -2
    assert call(r=33) == -2
    assert call(iters=0) == -7
    assert call(w=MIS) == -4
    assert call(gs=A + 2) == -4
    assert call(ws_bytes=ws - 1) == -5


def test_active_set_argument_errors():
    n = ctypes.c_int32()
    assert L.ffn_active_set(None, 1, 64, 128, 0, ctypes.byref(n), A, None, None) == -1
    assert L.ffn_active_set(A, 65, 64, 128, 0, ctypes.byref(n), A, None, None) == -2
    assert L.ffn_active_set(A, 1, 64, 128, -1, ctypes.byref(n), A, None, None) == -2


def test_timing_hook_argument_errors():
    assert L.ffn_time_next_gate_kernel(A, None) == -1
    assert L.ffn_time_next_gate_kernel(None, A) == -1
    assert L.ffn_time_next_gate_kernel(None, None) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(ffn, "_lib", None)
    monkeypatch.setattr(ffn, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        ffn.lib()


def test_workspace_active_pointers():
    """ffn_workspace_active is pointer arithmetic on the host: no device access, so it runs
    here; the views lie inside the workspace, in layout order, 256-byte aligned."""
    vp = ctypes.c_void_p
    for T, d, d_ff, r in ((1, 4096, 14336, 0), (4, 264, 1000, 40), (64, 136, 300, 0)):
        out = [vp() for _ in range(4)]
        assert L.ffn_workspace_active(A, T, d, d_ff, r, *(ctypes.byref(p) for p in out)) == 0
        meta, cnt, idx, act = (p.value for p in out)
        n = ffn.workspace_bytes(T, d, d_ff, r)
        assert A <= meta < cnt < idx < act and act + 4 * T * d_ff <= A + n
        assert cnt - meta >= 4 * 64 and idx - cnt >= 4 * d_ff and act - idx >= 4 * d_ff
        assert all((p - A) % 256 == 0 for p in (meta, cnt, idx, act))
    out = [vp() for _ in range(4)]
    refs = [ctypes.byref(p) for p in out]
    assert L.ffn_workspace_active(None, 1, 64, 128, 0, *refs) == -1
    assert L.ffn_workspace_active(A, 1, 64, 128, 0, None, *refs[1:]) == -1
    assert L.ffn_workspace_active(A, 0, 64, 128, 0, *refs) == -2
    assert L.ffn_workspace_active(A, 65, 64, 128, 0, *refs) == -2
    assert L.ffn_workspace_active(A, 1, 64, 128, -1, *refs) == -2


def test_noalloc_argument_errors():
    """The no-allocation entry point checks its arguments and its workspace limit before it
    touches the GPU."""
    f = L.ffn_sparse_forward_noalloc
    c = ctypes.c_float(0.5)
    assert f(1, 1, 64, 128, None, A, A, A, c, A, None) == -1
    assert f(1, 1, 64, 128, A, A, A, A, c, None, None) == -1
    assert f(7, 1, 64, 128, A, A, A, A, c, A, None) == -3
    assert f(1, 0, 64, 128, A, A, A, A, c, A, None) == -2
    assert f(1, 1, 64, 128, MIS, A, A, A, c, A, None) == -4
    assert ffn.workspace_bytes(64, 8192, 28672, 0) > 16 << 20
    assert f(1, 64, 8192, 28672, A, A, A, A, c, A, None) == -5


def test_z_wait_hook():
    """The test hook for the single-token LoPA kernel's bounded wait takes any tick count
    (host state only; nothing is launched)."""
    for ticks in (0, 1, 10000, (1 << 64) - 1):
        assert L.ffn_set_z_wait_ticks(ctypes.c_uint64(ticks)) == 0
    ffn.ffn_set_z_wait_ticks(ffn.Z_WAIT_TICKS_DEFAULT)
