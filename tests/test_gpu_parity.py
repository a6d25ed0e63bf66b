"""GPU parity: every entry point of the C ABI against the oracle on the same seeded
inputs (element-wise outputs, exact active sets outside the 1e-3 band).

Small shapes exercise every kernel variant with ragged tails; the full-size cases
are the workloads the benchmark times, in the same launch configuration.
"""
import numpy as np
import pytest

from paper_2609_31975_amd import workloads as wl

pytestmark = pytest.mark.gpu

F32, BF16 = wl.F32, wl.BF16


@pytest.fixture(scope="module")
def gu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from tests import gpu_util
    return gpu_util


# name, T, d, d_ff, r, wdt, t
SMALL = [
    ("tiny_f32_workload", 1, 256, 1024, 0, F32, 1.2816),   # the tiny fp32 workload, seed 0
    ("std_bf16_ragged", 1, 264, 1000, 0, BF16, 1.0),       # 33 chunks per row, last segment 8 rows
    ("std_bf16_long_rows", 1, 4104, 300, 0, BF16, 1.0),    # 513 chunks per row: 16 chunks per lane
    ("std_f32_ragged", 1, 260, 999, 0, F32, 0.8),
    ("std_bf16_odd_d", 1, 100, 77, 0, BF16, 0.5),          # d not a multiple of 8: element-wise kernels
    ("std_f32_odd_d", 1, 102, 130, 0, F32, 0.5),
    ("std_bf16_T3", 3, 264, 1000, 0, BF16, 1.0),           # union of 3 active sets
    ("std_f32_T70", 70, 64, 200, 0, F32, 1.0),             # two token passes (64 + 6)
    ("lopa_bf16", 1, 264, 1000, 40, BF16, 1.0),
    ("lopa_bf16_odd_r", 1, 264, 1000, 36, BF16, 1.0),
    ("lopa_f32", 1, 256, 1024, 32, F32, 1.2816),
    ("lopa_bf16_T5", 5, 264, 1000, 40, BF16, 1.0),
    ("std_bf16_T2", 2, 264, 1000, 0, BF16, 1.0),            # matrix-core gate, vector down (2 tokens)
    ("std_bf16_T8", 8, 264, 1000, 0, BF16, 1.2),
    ("std_bf16_T12", 12, 264, 1000, 0, BF16, 1.2),          # matrix-core down, one token tile
    ("lopa_bf16_T20", 20, 264, 1000, 40, BF16, 1.3),        # two token tiles
    ("std_bf16_T40", 40, 136, 300, 0, BF16, 1.5),           # four token tiles, short rows
    ("std_bf16_T64", 64, 264, 1000, 0, BF16, 1.6),
    ("std_bf16_T17", 17, 136, 300, 0, BF16, 1.2),           # pre-split tokens, second tile nearly empty
    ("std_bf16_T8_dff24576", 8, 264, 24576, 0, BF16, 1.2),  # 512 segments: two halves a gate workgroup
    ("lopa_bf16_T8_dff24576", 8, 264, 24576, 40, BF16, 1.2),  # LoPA with two gate workgroups a CU
    ("lopa_bf16_T16_dff24600", 16, 264, 24600, 72, BF16, 1.4),  # ragged segments, 16 tokens
    ("lopa_bf16_T70", 70, 264, 1000, 40, BF16, 1.3),        # a pre-split 64-token pass, then 6 tokens
    ("std_bf16_T100", 100, 264, 1000, 0, BF16, 1.6),        # 64 + 36: the tail pass is pre-split (three tiles)
    ("lopa_bf16_T100", 100, 264, 1000, 40, BF16, 1.6),
    ("lopa_bf16_T81", 81, 264, 1000, 40, BF16, 1.6),        # 64 + 17: a tail pass of two tiles, one token in the second
    ("std_bf16_d4096", 1, 4096, 2056, 0, BF16, 1.2816),    # full-width rows, short d_ff
    ("std_bf16_d4096_odd", 1, 4096, 2052, 0, BF16, 1.2816),
    ("std_bf16_long_chunks", 1, 4096, 40000, 0, BF16, 1.2816),  # down row chunks of over 1024 slots
    # one row per wave: W_up rows of active neurons interleaved with the gate stream
    ("std_bf16_d4096_half_active", 1, 4096, 2056, 0, BF16, 0.0),   # runs of consecutive active rows
    ("std_bf16_d4096_all_active", 1, 4096, 300, 0, BF16, -100.0),  # every gate row followed by its W_up row
    ("std_bf16_d4096_one_row_segs", 1, 4096, 100, 0, BF16, 0.0),   # segments of one row: idle waves
    ("std_bf16_d8192", 1, 8192, 1500, 0, BF16, 1.2816),            # one buffer a wave (16 chunks a lane)
    ("std_f32_d2048", 1, 2048, 1500, 0, F32, 1.2816),
    ("std_bf16_T4_odd_d", 4, 100, 77, 0, BF16, 0.5),       # batch with d not a multiple of 8: element-wise
    # 2..4 tokens, standard gating: the 4x4x4 matrix-core kernel (rows padded to 128 elements fit 4096)
    ("std_bf16_T4_q4_d4096", 4, 4096, 3000, 0, BF16, 1.2816),  # the largest d it takes; 63-row segments
    ("std_bf16_T3_q4_short", 3, 136, 77, 0, BF16, 0.5),        # 17 chunks: a step of one chunk; 2 segments
    ("std_bf16_T2_d4104", 2, 4104, 500, 0, BF16, 1.0),         # one step past its token LDS: 16x16x32 kernel
    ("lopa_bf16_T4_q4_r1024", 4, 4096, 3000, 1024, BF16, 1.2816),  # the largest r it takes
    ("lopa_bf16_T2_q4_r48", 2, 264, 1000, 48, BF16, 1.0),          # 6 chunks of z: one partial step
    ("lopa_bf16_T3_r1032", 3, 264, 500, 1032, BF16, 1.0),          # r past its z LDS: 16x16x32 kernel
    ("lopa_bf16_T3_odd_r", 3, 264, 1000, 36, BF16, 1.0),    # batch with r not a multiple of 8: element-wise
    ("very_small", 1, 8, 3, 0, BF16, 0.0),
    ("d_is_1", 1, 1, 5, 0, F32, 0.0),
    ("lopa_r_is_1", 2, 16, 40, 1, F32, 0.1),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
@pytest.mark.parametrize("dense", [False, True], ids=["sparse", "dense"])
def test_small_shapes(gu, case, dense):
    name, T, d, d_ff, r, wdt, t = case
    inp = wl.make_inputs(101, T, d, d_ff, r=r, wdt=wdt)
    dev = gu.DevInputs(inp)
    y, idx, act, _ = gu.run_gpu(dev, t, dense=dense)
    res = gu.run_oracle(inp, t, dense=dense)
    gu.check_parity(res, y, idx, act, t, wdt, dense=dense, what=name)


# ---------------------------------------------------------------- full-size workloads
_cache = {}


def _inputs(key, T, d, d_ff, r, seed):
    if key not in _cache:
        _cache.clear()
        _cache[key] = wl.make_inputs(seed, T, d, d_ff, r=r, wdt=BF16)
    return _cache[key]


# the full form and quantized weights have files of their own
FULL = [w for w in wl.workloads() if w.name != "tiny_f32_std_s90" and not w.form and w.wdt == BF16 and not w.rho]


@pytest.mark.parametrize("w", FULL, ids=[w.name for w in FULL])
def test_full_size_workloads(gu, w):
    inp = _inputs((w.d, w.d_ff, w.r, w.T, w.seed), w.T, w.d, w.d_ff, w.r, w.seed)
    dev = gu.DevInputs(inp)
    y, idx, act, _ = gu.run_gpu(dev, w.t)
    res = gu.run_oracle(inp, w.t)
    fig = gu.check_parity(res, y, idx, act, w.t, w.wdt, what=w.name)
    print(w.name, fig["max_rel_err"], fig["n_union"], fig["band_flips"], flush=True)


@pytest.mark.parametrize("r", [0, 512], ids=["standard", "lopa512"])
def test_full_size_dense(gu, r):
    inp = _inputs((4096, 14336, r, 1, 1000 + r), 1, 4096, 14336, r, 1000 + r)
    dev = gu.DevInputs(inp)
    y, idx, act, _ = gu.run_gpu(dev, 1.2816, dense=True)
    res = gu.run_oracle(inp, 1.2816, dense=True)
    gu.check_parity(res, y, idx, act, 1.2816, BF16, dense=True, what=f"dense r={r}")


# ---------------------------------------------------------------- edge cases
EDGE_SHAPES = [(1, 264, 1000, 0, BF16), (1, 100, 77, 0, BF16), (1, 264, 1000, 40, BF16), (4, 64, 200, 0, F32),
               (4, 264, 1000, 0, BF16), (16, 264, 1000, 40, BF16), (64, 136, 300, 0, BF16),  # matrix-core batches
               (1, 4096, 1000, 0, BF16)]  # full-width rows, few segments
POISON_SHAPES = EDGE_SHAPES[:3] + [(2, 264, 1000, 0, BF16), (2, 264, 1000, 40, BF16), (1, 4096, 1000, 0, BF16)]


@pytest.mark.parametrize("shape", EDGE_SHAPES, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}_w{s[4]}")
def test_nothing_active(gu, shape):
    T, d, d_ff, r, wdt = shape
    inp = wl.make_inputs(102, T, d, d_ff, r=r, wdt=wdt)
    y, idx, act, _ = gu.run_gpu(gu.DevInputs(inp), 1e30)
    assert len(idx) == 0 and np.all(y == 0)


@pytest.mark.parametrize("shape", EDGE_SHAPES, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}_w{s[4]}")
def test_everything_active_equals_dense(gu, shape):
    T, d, d_ff, r, wdt = shape
    inp = wl.make_inputs(103, T, d, d_ff, r=r, wdt=wdt)
    dev = gu.DevInputs(inp)
    ys, idx, _, _ = gu.run_gpu(dev, -100.0)
    yd, _, _, _ = gu.run_gpu(dev, -100.0, dense=True)
    assert idx.tolist() == list(range(d_ff))
    assert gu.rel_err(ys, yd) < 1e-6      # same terms; only the order of atomic additions differs
    gu.check_parity(gu.run_oracle(inp, -100.0), ys, None, None, -100.0, wdt)


@pytest.mark.parametrize("shape", POISON_SHAPES, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}")
def test_inactive_rows_are_never_read(gu, shape):
    """NaN in every W_up / W_down^T row that no token activates: the output is unchanged."""
    T, d, d_ff, r, wdt = shape
    inp = wl.make_inputs(104, T, d, d_ff, r=r, wdt=wdt)
    t = 1.0
    res = gu.run_oracle(inp, t)
    off = ~res.active.any(0)
    near = (np.abs(res.h - t) < gu.BAND).any(0)
    poison = off & ~near
    assert poison.sum() > d_ff // 2
    up, dn = inp.w_up.copy(), inp.w_down_t.copy()
    nan = np.uint16(0x7FC0) if wdt == BF16 else np.float32(np.nan)
    up[poison] = nan
    dn[poison] = nan
    pinp = wl.FFNInputs(x=inp.x, w_up=up, w_down_t=dn, w_gate=inp.w_gate, lopa_a=inp.lopa_a, lopa_b=inp.lopa_b,
                        wdt=wdt)
    y, idx, act, _ = gu.run_gpu(gu.DevInputs(pinp), t)
    assert np.isfinite(y).all()
    gu.check_parity(res, y, idx, act, t, wdt, what="poisoned")


# ---------------------------------------------------------------- one workspace, many shapes
# The header lets one workspace (zero-filled once, large enough) serve every later call: each
# call leaves it ready for the next, whatever the next one's shape.  The layout moves with the
# shape, so the regions of one call lie over other regions of the next; the single-token LoPA
# calls' tagged z words must still never read as published when they are not.
SHARED_WS = [(1, 1024, 3000, 512, BF16), (1, 1024, 3000, 0, BF16), (4, 1024, 3000, 512, BF16),
             (1, 1024, 3000, 256, BF16), (20, 1024, 3000, 0, BF16), (1, 1024, 3000, 1024, BF16),
             (1, 264, 1000, 40, F32), (70, 264, 1000, 40, BF16), (1, 1024, 3000, 512, wl.I8),
             (8, 1024, 3000, 512, BF16), (1, 1024, 3000, 512, BF16)]


def test_workspace_shared_across_shapes(gu):
    import torch
    from paper_2609_31975_amd import ffn
    t = 1.2816
    cases = [(shape, wl.make_inputs(120 + k, *shape[:3], r=shape[3], wdt=shape[4])) for k, shape in enumerate(SHARED_WS)]
    nbytes = max(ffn.workspace_bytes(T, d, d_ff, r) for (T, d, d_ff, r, _), _ in cases)
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    devs = [gu.DevInputs(inp) for _, inp in cases]
    refs = [gu.run_oracle(inp, t) for _, inp in cases]
    for rnd in range(2):
        for k, ((T, d, d_ff, r, wdt), inp) in enumerate(cases):
            dv = devs[k]
            y = torch.full((T, d), float("nan"), dtype=torch.float32, device="cuda")
            if wdt == wl.I8:
                sc = dv.scales_struct()
                ffn.ffn_lopa_sparse_forward_q(dv.x, dv.lopa_a, dv.lopa_b, dv.w_up, dv.w_down_t, sc, t, None, y, ws)
            elif r:
                ffn.ffn_lopa_sparse_forward(dv.x, dv.lopa_a, dv.lopa_b, dv.w_up, dv.w_down_t, t, y, ws)
            else:
                ffn.ffn_sparse_forward(dv.x, dv.w_gate, dv.w_up, dv.w_down_t, t, y, ws)
            torch.cuda.synchronize()
            idx, act = ffn.ffn_active_set(ws, T, d, d_ff, r) if T <= 64 else (None, None)
            gu.check_parity(refs[k], y.cpu().numpy(), idx, act, t, wdt,
                            what=f"shared workspace, round {rnd}, call {k} (T{T} d{d} d_ff{d_ff} r{r})")


# ---------------------------------------------------------------- degenerate shapes
# d = 1, one neuron, r = 1 and the like: y rests on a handful of neurons, so it is checked
# against the fp64 rebuild from the kernel's own activation values (gu.check_rebuilt), and the
# active sets and activation values against the oracle as everywhere else.
DEGENERATE = [(1, 1, 1, 0, F32, -1.0), (1, 1, 64, 0, BF16, 0.0), (5, 1, 300, 0, F32, 0.5),
              (1, 64, 1, 0, BF16, -1.0), (3, 32, 1, 1, F32, 0.0), (4, 264, 5, 1, BF16, 0.0),
              (64, 1, 100, 0, BF16, 0.0), (1, 8, 1000, 1, F32, 0.5), (16, 8, 64, 8, BF16, 0.0),
              (1, 4096, 1, 0, BF16, -1.0), (2, 16, 1, 0, wl.I8, -1.0), (3, 2, 7, 2, wl.I4, 0.0),
              (1, 1, 5000, 1, BF16, 1.2816), (33, 3, 7, 3, F32, 0.0)]


@pytest.mark.parametrize("shape", DEGENERATE, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}_w{s[4]}_t{s[5]}")
def test_degenerate_shapes(gu, shape):
    T, d, d_ff, r, wdt, t = shape
    inp = wl.make_inputs(108, T, d, d_ff, r=r, wdt=wdt)
    dev = gu.DevInputs(inp)
    y, idx, act, _ = gu.run_gpu_q(dev, t) if wdt in (wl.I8, wl.I4) else gu.run_gpu(dev, t)
    res = gu.run_oracle(inp, t)
    name = f"degenerate T{T} d{d} d_ff{d_ff} r{r}"
    assert np.isfinite(y).all(), f"{name}: non-finite output"
    gu.check_parity(res, y, idx, act, t, wdt, what=name, check_y=False)
    gu.check_rebuilt(inp, y, idx, act, wdt, what=name)


# Inf / NaN in the rows of an active neuron, on each dispatch path: the single-token kernels
# (bf16 standard, fp32 LoPA), the 4x4x4 and 16x16 matrix-core batches (the latter with
# pre-split tokens) and the element-wise batch kernels (d not a multiple of 8)
NONFINITE_SHAPES = [(1, 4096, 1000, 0, BF16), (1, 256, 1024, 32, F32), (4, 1024, 2000, 0, BF16),
                    (20, 512, 1500, 64, BF16), (3, 100, 700, 0, BF16)]


@pytest.mark.parametrize("where", ["down_inf", "up_nan"])
@pytest.mark.parametrize("shape", NONFINITE_SHAPES, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}_w{s[4]}")
def test_nonfinite_rows_of_active_neurons(gu, shape, where):
    """Non-finite values in a W_up / W_down^T row of a neuron that token 0 activates reach
    token 0's output: +Inf at one W_down^T entry makes that column non-finite (sign(zval) x
    Inf for one token), NaN across the W_up row makes the whole output row NaN.  A token that does not activate the
    neuron gets the oracle's value or a non-finite one there (a batch reads the row for the
    union); every other entry matches the oracle."""
    T, d, d_ff, r, wdt = shape
    inp = wl.make_inputs(107, T, d, d_ff, r=r, wdt=wdt)
    t = 1.0
    res = gu.run_oracle(inp, t)
    near = (np.abs(res.h - t) < gu.BAND).any(0)
    cand = np.flatnonzero(res.active[0] & ~near)
    assert cand.size, "no active neuron clear of the band"
    i, c = int(cand[cand.size // 2]), d // 3
    # zval of neuron i for every token, from the oracle: W_down^T with row i all ones, the rest 0
    ones = np.uint16(0x3F80) if wdt == BF16 else np.float32(1.0)
    dz = np.zeros_like(inp.w_down_t)
    dz[i] = ones
    zval = gu.run_oracle(wl.FFNInputs(**{**inp.__dict__, "w_down_t": dz}), t).y[:, 0]
    if where == "down_inf":
        dn = inp.w_down_t.copy()
        dn[i, c] = np.uint16(0x7F80) if wdt == BF16 else np.float32(np.inf)
        pinp = wl.FFNInputs(**{**inp.__dict__, "w_down_t": dn})
    else:
        up = inp.w_up.copy()
        up[i] = np.uint16(0x7FC0) if wdt == BF16 else np.float32(np.nan)
        pinp = wl.FFNInputs(**{**inp.__dict__, "w_up": up})
    y, idx, act, _ = gu.run_gpu(gu.DevInputs(pinp), t)
    tol = gu.TOL[wdt]
    on = res.active[:, i]
    assert on[0]
    for tau in range(T):
        ref = np.asarray(res.y[tau], np.float64)
        scale = float(np.max(np.abs(ref)))
        row = np.asarray(y[tau], np.float64)
        if where == "down_inf":
            rest = np.arange(d) != c
            if on[tau] and T == 1:  # fp32 products: zval x Inf
                assert row[c] == np.sign(zval[tau]) * np.inf, f"token {tau}: column {c} is {row[c]}"
            elif on[tau]:  # a batch may multiply Inf with zval's bf16 hi and lo parts: Inf or NaN
                assert not np.isfinite(row[c]), f"token {tau}: column {c} is {row[c]}"
            else:
                assert not np.isfinite(row[c]) or abs(row[c] - ref[c]) <= tol * scale
            assert np.isfinite(row[rest]).all(), f"token {tau}: non-finite outside column {c}"
            assert np.max(np.abs(row[rest] - ref[rest])) <= tol * scale
        elif on[tau]:
            assert np.isnan(row).all(), f"token {tau}: {np.isfinite(row).sum()} finite entries"
        else:
            assert np.isnan(row).all() or np.max(np.abs(row - ref)) <= tol * scale


@pytest.mark.parametrize("wdt", [F32, BF16])
def test_worked_example_on_gpu(gu, wdt):
    """The hand-worked example of the oracle pins (exact arithmetic; neuron 0 sits on the threshold)."""
    from tests.test_oracle import _enc, _worked_standard
    x, g, up, dn = _worked_standard()
    up = np.nan_to_num(up, nan=0.0)
    dn = np.nan_to_num(dn, nan=0.0)
    inp = wl.FFNInputs(x=x, w_gate=_enc(g, wdt), w_up=_enc(up, wdt), w_down_t=_enc(dn, wdt), wdt=wdt)
    y, idx, act, _ = gu.run_gpu(gu.DevInputs(inp), 1.0)
    assert y.tolist() == [[0.5, -2, -2, 15]]
    assert idx.tolist() == [1, 2, 5] and act.tolist() == [[1, 2, 5]]


@pytest.mark.parametrize("r", [0, 512])
def test_repeatable(gu, r):
    """Active set and activations are bit-identical across runs; y differs at most by
    the order of its fp32 atomic additions."""
    inp = wl.make_inputs(105, 1, 4096, 14336, r=r, wdt=BF16)
    dev = gu.DevInputs(inp)
    y1, i1, a1, _ = gu.run_gpu(dev, 1.2816)
    y2, i2, a2, _ = gu.run_gpu(dev, 1.2816)
    assert np.array_equal(i1, i2) and np.array_equal(a1.view(np.uint32), a2.view(np.uint32))
    assert gu.rel_err(y2, y1) < 1e-6


GRAPH_SHAPES = [(1, 4096, 2056, 0), (4, 264, 1000, 40), (20, 264, 1000, 40), (64, 264, 1000, 0),
                (1, 4096, 2056, 512),     # LoPA's z handed between gate workgroups through tagged words
                (3, 4096, 2056, 0), (3, 4096, 2056, 512),   # the 4x4x4 batch kernel
                (8, 1024, 24576, 0), (8, 1024, 24576, 64)]  # two gate workgroups a CU


@pytest.mark.parametrize("shape", GRAPH_SHAPES, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}")
def test_graph_replay(gu, shape):
    """A call captured in a HIP graph gives the eager result on every replay, with y
    filled with NaN and other eager work in between (y is fully overwritten each time)."""
    import torch
    from paper_2609_31975_amd import ffn
    T, d, d_ff, r = shape
    t = 1.2816
    inp = wl.make_inputs(107, T, d, d_ff, r=r, wdt=BF16)
    dev = gu.DevInputs(inp)
    ws = ffn.alloc_workspace(T, d, d_ff, r)
    y = torch.empty((T, d), dtype=torch.float32, device="cuda")

    def call():
        if r:
            ffn.ffn_lopa_sparse_forward(dev.x, dev.lopa_a, dev.lopa_b, dev.w_up, dev.w_down_t, t, y, ws)
        else:
            ffn.ffn_sparse_forward(dev.x, dev.w_gate, dev.w_up, dev.w_down_t, t, y, ws)

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        call()
    torch.cuda.synchronize()
    y_eager = y.cpu().numpy()
    gu.check_parity(gu.run_oracle(inp, t), y_eager, None, None, t, BF16, what="eager")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        call()
    other = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        y.fill_(float("nan"))
        other.mul_(1.0001)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        y_rep = y.cpu().numpy()
        assert np.isfinite(y_rep).all(), f"replay {rep} left entries unwritten"
        assert gu.rel_err(y_rep, y_eager) < 1e-6, f"replay {rep}"
    del graph


# ---------------------------------------------------------------- random shapes
def _random_cases(n=40, seed=2026):
    """Seeded shapes across every dispatch path: token counts 1..130 (several passes of 64),
    d and r multiples of 8 (fast and matrix-core kernels) or not (element-wise), short and
    ragged d_ff, at most about 2e8 multiply-adds for the oracle."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        i = len(cases)
        T = int(rng.choice([1, 1, 1, 2, 3, 4, 5, 8, 13, 16, 17, 33, 64, 70, 130]))
        d = int(rng.choice([8, 64, 136, 264, 520, 1032, 2056, 4096, 100, 250]))
        d_ff = int(rng.integers(3, 5000))
        r = int(rng.choice([0, 0, 0, 8, 16, 40, 24, 36, 128, 520]))
        if T * d * (d_ff + r) > 2e8:
            continue
        wdt = BF16 if rng.random() < 0.75 else F32
        t = float(rng.choice([0.0, 0.8416, 1.2816, 1.6449]))
        cases.append((f"rand{i}_T{T}_d{d}_dff{d_ff}_r{r}_{'bf16' if wdt == BF16 else 'f32'}", T, d, d_ff, r, wdt, t))
    return cases


RANDOM = _random_cases()


@pytest.mark.parametrize("case", RANDOM, ids=[c[0] for c in RANDOM])
def test_random_shapes(gu, case):
    name, T, d, d_ff, r, wdt, t = case
    inp = wl.make_inputs(106, T, d, d_ff, r=r, wdt=wdt)
    dev = gu.DevInputs(inp)
    y, idx, act, _ = gu.run_gpu(dev, t)
    gu.check_parity(gu.run_oracle(inp, t), y, idx, act, t, wdt, what=name)


# ---------------------------------------------------------------- correlated batches
@pytest.mark.parametrize("rho", [0.5, 0.9, 1.0])
@pytest.mark.parametrize("T,r", [(16, 512), (64, 512), (20, 0)])
def test_correlated_batches(gu, rho, T, r):
    """Tokens sharing a common part (the union shrinks as rho grows; rho = 1: T identical
    tokens, one active set)."""
    d, d_ff = 4096, 14336 if r else 3000
    inp = _inputs((d, d_ff, r, T, 3000 + r), T, d, d_ff, r, 3000 + r)
    x = wl.make_tokens_correlated(71, T, d, rho)
    tch = __import__("torch")
    y, idx, act, _ = gu.run_gpu(gu.DevInputs(inp), 1.2816, x=tch.from_numpy(x).to("cuda"))
    res = gu.run_oracle(inp, 1.2816, x=x)
    fig = gu.check_parity(res, y, idx, act, 1.2816, BF16, what=f"rho={rho} T={T} r={r}")
    n1 = np.mean(fig["n_active"])
    assert n1 <= fig["n_union"] <= T * n1
    if rho == 1.0:
        assert fig["n_union"] == round(n1)
    print(f"rho={rho} T={T} r={r}: union {fig['n_union']} of {d_ff}, per token {n1:.0f}", flush=True)


# ---------------------------------------------------------------- NaN gate values
NAN_GATE = [(1, 264, 1000, 0, BF16), (1, 260, 999, 0, F32), (4, 264, 1000, 0, BF16), (4, 264, 1000, 0, F32),
            (1, 264, 1000, 40, BF16), (1, 256, 1024, 32, F32), (4, 264, 1000, 40, BF16), (4, 264, 1000, 40, F32),
            (1, 4096, 2056, 0, BF16)]


@pytest.mark.parametrize("shape", NAN_GATE, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}_w{s[4]}")
def test_nan_gate_rows_are_inactive(gu, shape):
    """NaN in a few W_gate rows (or B rows for LoPA) makes those gate values NaN: the
    neurons are inactive (h > t is false), the rest of the call is unaffected and y is
    finite."""
    T, d, d_ff, r, wdt = shape
    inp = wl.make_inputs(108, T, d, d_ff, r=r, wdt=wdt)
    nan = np.uint16(0x7FC0) if wdt == BF16 else np.float32(np.nan)
    rows = np.arange(3, d_ff, 97)
    if r:
        inp.lopa_b = inp.lopa_b.copy()
        inp.lopa_b[rows] = nan
    else:
        inp.w_gate = inp.w_gate.copy()
        inp.w_gate[rows] = nan
    t = 0.9
    res = gu.run_oracle(inp, t)
    assert np.isnan(res.h[:, rows]).all() and not res.active[:, rows].any()
    y, idx, act, _ = gu.run_gpu(gu.DevInputs(inp), t)
    assert np.isfinite(y).all()
    assert not np.isin(rows, idx).any(), "a NaN gate value was listed as active"
    gu.check_parity(res, y, idx, act, t, wdt, what=f"nan gate {shape}")


# ---------------------------------------------------------------- device views of the active set
@pytest.mark.parametrize("shape", [(1, 4096, 2056, 0), (1, 264, 1000, 40), (4, 264, 1000, 40), (20, 264, 1000, 0)],
                         ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}")
def test_workspace_active_under_graph_capture(gu, shape):
    """ffn_workspace_active gives device pointers into the workspace without synchronizing:
    a graph that holds the call and copies of those views (device work reading them right
    after the call) replays, for new tokens each time, to the active set that the
    synchronizing host hook reports."""
    import torch
    from paper_2609_31975_amd import ffn
    T, d, d_ff, r = shape
    t = 1.2816
    inp = wl.make_inputs(109, T, d, d_ff, r=r, wdt=BF16)
    dev = gu.DevInputs(inp)
    ws = ffn.alloc_workspace(T, d, d_ff, r)
    y = torch.empty((T, d), dtype=torch.float32, device="cuda")
    x = dev.x.clone()
    meta, cnt, idx, act = ffn.ffn_workspace_active(ws, T, d, d_ff, r)

    def call():
        if r:
            ffn.ffn_lopa_sparse_forward(x, dev.lopa_a, dev.lopa_b, dev.w_up, dev.w_down_t, t, y, ws)
        else:
            ffn.ffn_sparse_forward(x, dev.w_gate, dev.w_up, dev.w_down_t, t, y, ws)

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        call()   # eager warm-up (kernel loading, occupancy queries)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        call()
        got = [v.clone() for v in (meta, cnt, idx, act)]
    for rep in range(3):
        x.copy_(torch.from_numpy(wl.make_tokens(110 + rep, T, d)).to("cuda"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        m, c, ix, a = (v.cpu().numpy() for v in got)
        nseg = int(m[0])
        assert 1 <= nseg <= d_ff
        q, rem = divmod(d_ff, nseg)
        starts = [w * q + min(w, rem) for w in range(nseg)]
        listed = np.concatenate([ix[s:s + c[w]] for w, s in enumerate(starts)])
        acts = np.concatenate([a[:, s:s + c[w]] for w, s in enumerate(starts)], axis=1)
        ref_idx, ref_act = ffn.ffn_active_set(ws, T, d, d_ff, r)
        assert np.array_equal(listed, ref_idx), f"replay {rep}"
        assert np.array_equal(acts.view(np.uint32), ref_act.view(np.uint32)), f"replay {rep}"
        res = gu.run_oracle(inp, t, x=x.cpu().numpy())
        gu.check_parity(res, y.cpu().numpy(), listed, acts, t, BF16, what=f"graph replay {rep}")
    del graph


# ---------------------------------------------------------------- LoPA's z, computed by each workgroup
# The single-token LoPA gate kernel shares z = A x between its workgroups and, past a bounded
# wait, has a workgroup compute the components it has not seen itself.  A wait of 0 ticks (set
# from the host; every kernel still ends normally) sends most workgroups down that path.
Z_SELF = [
    ("bf16_small", 264, 1000, 40, BF16, 1.0, False),
    ("f32_small", 256, 1024, 32, F32, 1.2816, False),
    ("bf16_8b_r512", 4096, 14336, 512, BF16, 1.2816, False),
    ("bf16_70b_r1024", 8192, 2048, 1024, BF16, 1.2816, False),
    ("bf16_norm_g", 264, 1000, 40, BF16, 1.0 * 2 ** 0.5, True),   # RMSNorm and G after the wait
]


@pytest.mark.parametrize("case", Z_SELF, ids=[c[0] for c in Z_SELF])
def test_lopa_z_computed_by_each_workgroup(gu, case):
    from paper_2609_31975_amd import ffn
    name, d, d_ff, r, wdt, t, full = case
    inp = wl.make_inputs(303, 1, d, d_ff, r=r, wdt=wdt)
    dev = gu.DevInputs(inp)
    form = None
    if full:
        form = gu.Form(act=1, silu_up=True, form=wl.make_form(304, d, d_ff, r), use_g=True, rms_norm=True,
                       use_gain=True)
    ffn.ffn_set_z_wait_ticks(0)
    try:
        if form is None:
            y, idx, act, _ = gu.run_gpu(dev, t)
        else:
            y, idx, act, _ = gu.run_gpu_ex(dev, t, form)
    finally:
        ffn.ffn_set_z_wait_ticks(ffn.Z_WAIT_TICKS_DEFAULT)
    res = gu.run_oracle(inp, t, form=form)
    gu.check_parity(res, y, idx, act, t, wdt, what=f"z computed by each workgroup, {name}",
                    act_value=None if form is None else form.act_value)
    # and the default wait again on the same inputs
    y2, idx2, act2, _ = gu.run_gpu(dev, t) if form is None else gu.run_gpu_ex(dev, t, form)
    gu.check_parity(res, y2, idx2, act2, t, wdt, what=f"default wait, {name}",
                    act_value=None if form is None else form.act_value)


# ---------------------------------------------------------------- graph replay: full form, int8 codes
@pytest.mark.parametrize("kind,T,r", [("form", 1, 512), ("form", 4, 512), ("form", 20, 40), ("int8", 1, 0),
                                      ("int8", 1, 512), ("int8", 4, 512), ("int4", 16, 64)])
def test_graph_replay_form_and_codes(gu, kind, T, r):
    """The full form (G, RMSNorm, R-S+, SiLU) and int8 / int4 codes captured in a HIP graph:
    every replay gives the eager result, with y filled with NaN and other work in between."""
    import torch
    from paper_2609_31975_amd import ffn
    d, d_ff = (4096, 2056) if T <= 4 else (264, 1000)
    wdt = {"form": BF16, "int8": wl.I8, "int4": wl.I4}[kind]
    inp = wl.make_inputs(108, T, d, d_ff, r=r, wdt=wdt)
    dev = gu.DevInputs(inp)
    form = None
    t = 1.2816
    if kind == "form":
        form = gu.Form(act=1, silu_up=True, form=wl.make_form(109, d, d_ff, r), use_g=True, rms_norm=True,
                       use_gain=True)
        t *= 2 ** 0.5
    ws = ffn.alloc_workspace(T, d, d_ff, r)
    y = torch.empty((T, d), dtype=torch.float32, device="cuda")
    opt = None if form is None else form.options()
    sc = None if kind == "form" else dev.scales_struct()
    gate = (dev.lopa_a, dev.lopa_b) if r else (dev.w_gate,)

    def call():
        if kind == "form":
            fn = ffn.ffn_lopa_sparse_forward_ex if r else ffn.ffn_sparse_forward_ex
            fn(dev.x, *gate, dev.w_up, dev.w_down_t, t, opt, y, ws)
        else:
            fn = ffn.ffn_lopa_sparse_forward_q if r else ffn.ffn_sparse_forward_q
            fn(dev.x, *gate, dev.w_up, dev.w_down_t, sc, t, opt, y, ws)

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        call()
    torch.cuda.synchronize()
    y_eager = y.cpu().numpy()
    gu.check_parity(gu.run_oracle(inp, t, form=form), y_eager, None, None, t, wdt, what=f"{kind} eager")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        call()
    other = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        y.fill_(float("nan"))
        other.mul_(1.0001)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        y_rep = y.cpu().numpy()
        assert np.isfinite(y_rep).all(), f"replay {rep} left entries unwritten"
        assert gu.rel_err(y_rep, y_eager) < 1e-6, f"replay {rep}"
    del graph


# ---------------------------------------------------------------- concurrent calls
@pytest.mark.parametrize("r", [0, 512], ids=["standard", "lopa512"])
def test_concurrent_streams(gu, r):
    """Calls with distinct workspaces on two streams at once (the header allows it): each
    stream's results equal a call made alone.  With LoPA, the two single-token gate kernels
    share the GPU, so their workgroups are not all resident together and the bounded wait
    for z (each workgroup computing what it has not seen) keeps both finite."""
    import torch
    from paper_2609_31975_amd import ffn
    d, d_ff, t = 4096, 14336, 1.2816
    inps = [wl.make_inputs(110 + k, 1, d, d_ff, r=r, wdt=BF16) for k in range(2)]
    devs = [gu.DevInputs(i) for i in inps]
    wss = [ffn.alloc_workspace(1, d, d_ff, r) for _ in range(2)]
    ys = [torch.empty((1, d), dtype=torch.float32, device="cuda") for _ in range(2)]

    def call(k):
        dv = devs[k]
        if r:
            ffn.ffn_lopa_sparse_forward(dv.x, dv.lopa_a, dv.lopa_b, dv.w_up, dv.w_down_t, t, ys[k], wss[k])
        else:
            ffn.ffn_sparse_forward(dv.x, dv.w_gate, dv.w_up, dv.w_down_t, t, ys[k], wss[k])

    alone = []
    for k in range(2):
        call(k)
        torch.cuda.synchronize()
        alone.append(ys[k].cpu().numpy())
        gu.check_parity(gu.run_oracle(inps[k], t), alone[k], None, None, t, BF16, what=f"alone {k}")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(20):
        for k in range(2):
            ys[k].fill_(float("nan"))
        torch.cuda.synchronize()
        for k in range(2):
            with torch.cuda.stream(streams[k]):
                call(k)
        torch.cuda.synchronize()
        for k in range(2):
            got = ys[k].cpu().numpy()
            assert np.isfinite(got).all(), f"rep {rep} stream {k}: entries unwritten"
            assert gu.rel_err(got, alone[k]) < 1e-5, f"rep {rep} stream {k}"
