"""GPU parity of weight-only int8 / int4 weights (the ``_q`` entry points) against the
oracle on the same codes and row scales: the single-token kernels (integer dot products
against a fixed-point copy of x or z) at one and two chunk groups per lane, the
element-wise kernels for other shapes and for batches, the full form on top, and the
benchmarked 8B workloads.
"""
import math

import numpy as np
import pytest

from paper_2609_31975_amd import workloads as wl

pytestmark = pytest.mark.gpu

I8, I4 = wl.I8, wl.I4


@pytest.fixture(scope="module")
def gu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from tests import gpu_util
    return gpu_util


# name, T, d, d_ff, r, wdt, t
SMALL = [
    ("i8_t1_std", 1, 256, 1000, 0, I8, 1.0),            # 16 chunks a row: 4 lanes a row
    ("i8_t1_std_d4096", 1, 4096, 2056, 0, I8, 1.2816),  # 64 lanes a row, 4 chunks a lane
    ("i8_t1_std_d8192", 1, 8192, 600, 0, I8, 1.2816),   # 8 chunks a lane
    ("i4_t1_std", 1, 256, 1000, 0, I4, 1.0),
    ("i4_t1_std_d4096", 1, 4096, 2056, 0, I4, 1.2816),  # 2 chunks a lane
    ("i4_t1_std_d8192", 1, 8192, 600, 0, I4, 1.2816),   # 4 chunks a lane
    ("i8_t1_ragged", 1, 272, 999, 0, I8, 0.9),          # 17 chunks: a partly filled lane group
    ("i8_t1_long_chunks", 1, 4096, 40000, 0, I8, 1.2816),  # down row chunks of over 1024 slots
    ("i4_t1_long_chunks", 1, 4096, 40000, 64, I4, 1.2816),
    ("i4_t1_ragged", 1, 288, 999, 0, I4, 0.9),          # 9 chunks
    ("i8_t1_lopa", 1, 256, 1000, 32, I8, 1.0),
    ("i4_t1_lopa", 1, 256, 1000, 64, I4, 1.0),
    ("i8_t1_lopa_d4096", 1, 4096, 3000, 512, I8, 1.2816),
    ("i4_t1_lopa_d4096", 1, 4096, 3000, 512, I4, 1.2816),
    ("i8_gen_lopa_r40", 1, 256, 1000, 40, I8, 1.0),     # r not a multiple of 16: element-wise
    ("i8_gen_odd_d", 1, 100, 77, 0, I8, 0.5),
    ("i4_gen_even_d", 1, 102, 77, 0, I4, 0.5),          # d even, not a multiple of 32
    ("i8_T3", 3, 256, 1000, 0, I8, 1.0),                # batches: matrix cores, codes as bf16
    ("i4_T4_q4_d4096", 4, 4096, 3000, 0, I4, 1.2816),   # 4x4x4 kernel: 8 products a loaded chunk
    ("i8_T2_q4_ragged", 2, 272, 999, 0, I8, 0.9),       # 17 chunks: a step of one chunk
    ("i4_T3_q4_ragged", 3, 288, 999, 0, I4, 0.9),       # 9 chunks: one partial step
    ("i4_T4_q4_lopa_r512", 4, 4096, 3000, 512, I4, 1.2816),
    ("i8_T3_q4_lopa_r48", 3, 256, 1000, 48, I8, 1.0),   # three 16-code chunks of z
    ("i4_T5_lopa", 5, 256, 1000, 32, I4, 1.0),
    ("i8_T70", 70, 64, 200, 0, I8, 1.0),                # two token passes
    ("i8_T16_lopa", 16, 256, 1000, 32, I8, 1.0),
    ("i8_T2_lopa_r48", 2, 256, 1000, 48, I8, 1.0),      # r = 48: three 16-element chunks a B row
    ("i4_T20", 20, 288, 999, 0, I4, 0.9),               # two token tiles; 9 chunks a row
    ("i8_T40_ragged", 40, 272, 999, 0, I8, 0.9),        # pre-split tokens; a half k step at the end
    ("i4_T64_lopa", 64, 256, 1000, 64, I4, 1.0),        # four token tiles
    ("i8_T8_lopa_dff24576", 8, 256, 24576, 32, I8, 1.0),  # LoPA with two gate workgroups a CU
    ("i4_T6_std_dff24600", 6, 288, 24600, 0, I4, 0.9),    # the same for standard gating
    ("i8_T4_gen_odd_d", 4, 100, 77, 0, I8, 0.5),        # d not a multiple of 16: element-wise
    ("i4_T6_gen_d48", 6, 48, 77, 0, I4, 0.5),           # d not a multiple of 32: element-wise
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
@pytest.mark.parametrize("dense", [False, True], ids=["sparse", "dense"])
def test_quant_small(gu, case, dense):
    name, T, d, d_ff, r, wdt, t = case
    inp = wl.make_inputs(301, T, d, d_ff, r=r, wdt=wdt)
    y, idx, act, _ = gu.run_gpu_q(gu.DevInputs(inp), t, dense=dense)
    res = gu.run_oracle(inp, t, dense=dense)
    gu.check_parity(res, y, idx, act, t, wdt, dense=dense, what=name)


ALL = dict(act=1, silu_up=True, use_g=True, rms_norm=True, use_gain=True)
FORM_CASES = [("i8_t1_lopa_all", 1, 4096, 3000, 512, I8), ("i4_t1_lopa_all", 1, 4096, 3000, 512, I4),
              ("i8_t1_std_act", 1, 4096, 3000, 0, I8), ("i4_T3_lopa_all", 3, 256, 1000, 32, I4),
              ("i8_T4_std_act", 4, 4096, 3000, 0, I8)]


@pytest.mark.parametrize("case", FORM_CASES, ids=[c[0] for c in FORM_CASES])
def test_quant_full_form(gu, case):
    name, T, d, d_ff, r, wdt = case
    inp = wl.make_inputs(302, T, d, d_ff, r=r, wdt=wdt)
    flags = ALL if r else dict(act=1, silu_up=True)
    form = gu.Form(form=wl.make_form(9, d, d_ff, r), **flags)
    t = 1.2816 * (math.sqrt(2) if r else 1.0)
    y, idx, act, _ = gu.run_gpu_q(gu.DevInputs(inp), t, form=form)
    res = gu.run_oracle(inp, t, form=form)
    gu.check_parity(res, y, idx, act, t, wdt, what=name, act_value=form.act_value)


@pytest.mark.parametrize("wdt", [I8, I4], ids=["i8", "i4"])
@pytest.mark.parametrize("r", [0, 32], ids=["std", "lopa"])
def test_quant_inactive_rows_are_never_read(gu, wdt, r):
    """NaN row scales on every W_up / W_down^T row no token activates (single token)."""
    inp = wl.make_inputs(303, 1, 256, 1000, r=r, wdt=wdt)
    t = 1.0
    res = gu.run_oracle(inp, t)
    near = np.abs(res.h[0] - t) < gu.BAND
    poison = ~res.active[0] & ~near
    assert poison.sum() > 500
    sc = dict(inp.scales)
    sc["up"] = np.where(poison, np.float32(np.nan), sc["up"]).astype(np.float32)
    sc["down"] = np.where(poison, np.float32(np.nan), sc["down"]).astype(np.float32)
    pois = wl.FFNInputs(**{**inp.__dict__, "scales": sc})
    y, idx, act, _ = gu.run_gpu_q(gu.DevInputs(pois), t)
    gu.check_parity(gu.run_oracle(pois, t), y, idx, act, t, wdt, what="poisoned")


@pytest.mark.parametrize("wdt", [I8, I4], ids=["i8", "i4"])
def test_quant_degenerate_thresholds(gu, wdt):
    inp = wl.make_inputs(304, 1, 4096, 600, r=0, wdt=wdt)
    dev = gu.DevInputs(inp)
    y, idx, _, _ = gu.run_gpu_q(dev, 1e30)
    assert len(idx) == 0 and np.all(y == 0)
    ys, idx, _, _ = gu.run_gpu_q(dev, -100.0)
    yd, _, _, _ = gu.run_gpu_q(dev, -100.0, dense=True)
    assert idx.tolist() == list(range(600)) and gu.rel_err(ys, yd) < 1e-6


@pytest.mark.parametrize("r", [0, 64], ids=["standard", "lopa64"])
def test_quant_zero_and_nonfinite_tokens(gu, r):
    """An all-zero token gives y = 0 with nothing active (the fixed-point scale of x, or z,
    is 0); a NaN in the token makes every gate value NaN, so nothing is active either."""
    inp = wl.make_inputs(305, 1, 4096, 600, r=r, wdt=I8)
    z = wl.FFNInputs(**{**inp.__dict__, "x": np.zeros_like(inp.x)})
    y, idx, _, _ = gu.run_gpu_q(gu.DevInputs(z), 0.0)
    assert len(idx) == 0 and np.all(y == 0)
    xn = inp.x.copy()
    xn[0, 7] = np.nan
    n = wl.FFNInputs(**{**inp.__dict__, "x": xn})
    y, idx, _, _ = gu.run_gpu_q(gu.DevInputs(n), 0.0)
    assert len(idx) == 0


QW = [w for w in wl.workloads() if w.wdt in (I8, I4)]


@pytest.mark.parametrize("w", QW, ids=[w.name for w in QW])
def test_quant_workloads(gu, w):
    inp = wl.make_inputs(w.seed, w.T, w.d, w.d_ff, r=w.r, wdt=w.wdt)
    y, idx, act, _ = gu.run_gpu_q(gu.DevInputs(inp), w.t)
    res = gu.run_oracle(inp, w.t)
    fig = gu.check_parity(res, y, idx, act, w.t, w.wdt, what=w.name)
    frac = np.mean(fig["n_active"]) / w.d_ff
    assert 0.05 < frac < 0.15
    print(w.name, fig["max_rel_err"], fig["n_union"], flush=True)


def _random_quant_cases(n=24, seed=2027):
    """Seeded shapes for int8 / int4 codes across the dispatch paths: d and r multiples of
    the chunk width (16 / 32 codes: integer-dot and matrix-core kernels) or only even
    (element-wise), 1..70 tokens, with and without the full form."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        i = len(cases)
        wdt = I8 if rng.random() < 0.5 else I4
        T = int(rng.choice([1, 1, 1, 2, 3, 4, 5, 8, 16, 17, 40, 70]))
        d = int(rng.choice([32, 64, 256, 512, 1024, 4096, 96, 100, 258]))
        d_ff = int(rng.integers(5, 4000))
        r = int(rng.choice([0, 0, 32, 64, 128, 512, 96, 34]))
        full = bool(rng.random() < 0.3)
        if T * d * (d_ff + r) > 2e8:
            continue
        tag = f"qrand{i}_{'i8' if wdt == I8 else 'i4'}_T{T}_d{d}_dff{d_ff}_r{r}{'_form' if full else ''}"
        cases.append((tag, T, d, d_ff, r, wdt, full))
    return cases


QRANDOM = _random_quant_cases()


@pytest.mark.parametrize("case", QRANDOM, ids=[c[0] for c in QRANDOM])
def test_quant_random_shapes(gu, case):
    name, T, d, d_ff, r, wdt, full = case
    inp = wl.make_inputs(305, T, d, d_ff, r=r, wdt=wdt)
    form = None
    t = 1.2816
    if full:
        flags = ALL if r else dict(act=1, silu_up=True)
        form = gu.Form(form=wl.make_form(10, d, d_ff, r), **flags)
        t *= math.sqrt(2) if r else 1.0
    y, idx, act, _ = gu.run_gpu_q(gu.DevInputs(inp), t, form=form)
    res = gu.run_oracle(inp, t, form=form)
    gu.check_parity(res, y, idx, act, t, wdt, what=name, act_value=None if form is None else form.act_value)
