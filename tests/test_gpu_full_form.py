"""GPU parity of the paper's full FFN form (the ``_ex`` entry points) against the oracle:
the R-S+ activation value, SiLU on the W_up output (the double activation of
Section 3.3), LoPA's fixed term G and RMSNorm between the LoPA factors (Section 3.3,
Eq. (lopaapprox)).  Every kernel family runs: the single-token kernels, the
element-wise kernels (odd d or r), and the matrix-core batch path at one, two and
four token tiles, with and without pre-split tokens.
"""
import math

import numpy as np
import pytest

from paper_2609_31975_amd import workloads as wl

pytestmark = pytest.mark.gpu

F32, BF16 = wl.F32, wl.BF16
S2 = math.sqrt(2.0)   # G adds a unit-variance term to the gate


@pytest.fixture(scope="module")
def gu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from tests import gpu_util
    return gpu_util


ACT = dict(act=1, silu_up=True)                                  # activations only
ALL = dict(act=1, silu_up=True, use_g=True, rms_norm=True, use_gain=True)
G_ONLY = dict(use_g=True)
NORM_ONLY = dict(rms_norm=True)

# name, T, d, d_ff, r, wdt, t, form flags
CASES = [
    ("t1_std_bf16_act", 1, 264, 1000, 0, BF16, 1.0, ACT),
    ("t1_std_f32_rsplus", 1, 260, 999, 0, F32, 0.8, dict(act=1)),
    ("t1_std_bf16_silu_d4096", 1, 4096, 2056, 0, BF16, 1.2816, dict(silu_up=True)),
    ("t1_lopa_bf16_all", 1, 264, 1000, 40, BF16, 1.0 * S2, ALL),
    ("t1_lopa_bf16_g", 1, 264, 1000, 40, BF16, 1.0 * S2, G_ONLY),
    ("t1_lopa_bf16_norm", 1, 264, 1000, 40, BF16, 1.0, NORM_ONLY),
    ("t1_lopa_f32_all", 1, 256, 1024, 32, F32, 1.2816 * S2, ALL),
    ("gen_std_bf16_odd_d", 1, 100, 77, 0, BF16, 0.5, ACT),
    ("gen_lopa_bf16_odd_r_T3", 3, 264, 1000, 36, BF16, 1.0 * S2, ALL),
    ("gen_lopa_f32_r1_T2", 2, 16, 40, 1, F32, 0.1, ALL),
    ("gen_std_f32_T70", 70, 64, 200, 0, F32, 1.0, ACT),
    ("mc_std_bf16_T2", 2, 264, 1000, 0, BF16, 1.0, ACT),
    ("q4_std_bf16_T4_act_d4096", 4, 4096, 3000, 0, BF16, 1.2816, ACT),
    ("q4_std_bf16_T3_silu", 3, 136, 77, 0, BF16, 0.5, dict(silu_up=True)),
    ("mc_std_bf16_T12", 12, 264, 1000, 0, BF16, 1.2, ACT),
    ("mc_lopa_bf16_T4_all", 4, 264, 1000, 40, BF16, 1.2 * S2, ALL),
    ("mc_lopa_bf16_T8_norm", 8, 264, 1000, 40, BF16, 1.2, NORM_ONLY),
    ("mc_lopa_bf16_T20_all", 20, 264, 1000, 40, BF16, 1.3 * S2, ALL),
    ("mc_std_bf16_T40", 40, 136, 300, 0, BF16, 1.5, ACT),
    ("mc_lopa_bf16_T64_all", 64, 264, 1000, 40, BF16, 1.6 * S2, ALL),
    ("mc_lopa_bf16_T70_g", 70, 264, 1000, 40, BF16, 1.3 * S2, dict(act=1, use_g=True)),
    ("mc_lopa_bf16_T90_all", 90, 264, 1000, 40, BF16, 1.6 * S2, ALL),   # 64 + 26: a pre-split two-tile tail
    ("mc_std_bf16_T100_act", 100, 264, 1000, 0, BF16, 1.6, ACT),
    ("mc2_lopa_bf16_T8_all", 8, 264, 24576, 40, BF16, 1.2 * S2, ALL),   # LoPA with two gate workgroups a CU
    ("mc2_std_bf16_T5_act", 5, 264, 24576, 0, BF16, 1.2, ACT),
]


def _form(gu, inp, flags):
    return gu.Form(form=wl.make_form(7, inp.d, inp.d_ff, inp.r), **flags)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("dense", [False, True], ids=["sparse", "dense"])
def test_full_form_small(gu, case, dense):
    name, T, d, d_ff, r, wdt, t, flags = case
    inp = wl.make_inputs(201, T, d, d_ff, r=r, wdt=wdt)
    form = _form(gu, inp, flags)
    y, idx, act, _ = gu.run_gpu_ex(gu.DevInputs(inp), t, form, dense=dense)
    res = gu.run_oracle(inp, t, dense=dense, form=form)
    fig = gu.check_parity(res, y, idx, act, t, wdt, dense=dense, what=name, act_value=form.act_value)
    if not dense and idx is not None:
        assert 0 < fig["n_union"] < d_ff or T > 8, f"{name}: degenerate active set"


def test_default_options_match_plain_calls(gu):
    """A zero-filled option struct is the default form: same result as the plain call."""
    for T, r in ((1, 0), (1, 40), (16, 40), (40, 0)):
        inp = wl.make_inputs(202, T, 264, 1000, r=r, wdt=BF16)
        dev = gu.DevInputs(inp)
        y0, idx0, _, _ = gu.run_gpu(dev, 1.0)
        y1, idx1, _, _ = gu.run_gpu_ex(dev, 1.0, gu.Form())
        assert np.array_equal(idx0, idx1)
        assert gu.rel_err(y1, y0) < 1e-6   # only the order of atomic additions differs


def test_same_active_set_for_either_activation(gu):
    """R-S+ and ReLU keep the same neurons (h > t); only their values differ."""
    inp = wl.make_inputs(203, 4, 264, 1000, r=40, wdt=BF16)
    dev = gu.DevInputs(inp)
    fi = wl.make_form(7, inp.d, inp.d_ff, inp.r)
    _, i0, a0, _ = gu.run_gpu_ex(dev, 1.3, gu.Form(form=fi, use_g=True))
    _, i1, a1, _ = gu.run_gpu_ex(dev, 1.3, gu.Form(act=1, form=fi, use_g=True))
    assert np.array_equal(i0, i1)
    assert np.array_equal(a0 > 0, a1 > 0)
    on = a0 > 0
    np.testing.assert_allclose(a1[on], a0[on] / (1.0 + np.exp(-a0[on].astype(np.float64))), rtol=1e-5)


# ---------------------------------------------------------------- full size: the benchmarked full-form workloads
FULL_FORM = [w for w in wl.workloads() if w.form == "full"]


@pytest.mark.parametrize("w", FULL_FORM, ids=[w.name for w in FULL_FORM])
def test_full_form_workloads(gu, w):
    inp = wl.make_inputs(w.seed, w.T, w.d, w.d_ff, r=w.r, wdt=w.wdt)
    form = gu.Form(form=wl.make_form(w.seed, w.d, w.d_ff, w.r), **ALL)
    y, idx, act, _ = gu.run_gpu_ex(gu.DevInputs(inp), w.t, form)
    res = gu.run_oracle(inp, w.t, form=form)
    fig = gu.check_parity(res, y, idx, act, w.t, w.wdt, what=w.name, act_value=form.act_value)
    frac = np.mean(fig["n_active"]) / w.d_ff
    assert 0.05 < frac < 0.15, f"activation fraction {frac:.3f} far from the 10% the threshold targets"
    print(w.name, fig["max_rel_err"], fig["n_union"], frac, flush=True)


# ---------------------------------------------------------------- s_gated: zero gated values
# (T, d, d_ff, r, wdt): the single-token kernels and the element-wise kernels (any T).  The
# matrix-core batch path multiplies every union row by every token's gated value.
SGATED = [(1, 264, 1000, 0, BF16), (1, 264, 1000, 40, BF16), (1, 260, 999, 0, F32), (1, 100, 77, 0, BF16),
          (3, 100, 77, 0, BF16), (4, 64, 200, 0, F32), (2, 264, 1000, 40, F32)]


@pytest.mark.parametrize("shape", SGATED, ids=lambda s: f"T{s[0]}_d{s[1]}_dff{s[2]}_r{s[3]}_w{s[4]}")
@pytest.mark.parametrize("silu_up", [False, True], ids=["plain", "silu"])
def test_zero_gated_value_rows_not_read(gu, shape, silu_up):
    """Active neurons with a zero W_up row have gated value 0: NaN in their W_down rows
    leaves the output equal to the oracle's (which skips those rows too)."""
    T, d, d_ff, r, wdt = shape
    inp = wl.make_inputs(205, T, d, d_ff, r=r, wdt=wdt)
    t = 0.8
    form = gu.Form(silu_up=silu_up)
    on = np.flatnonzero(gu.run_oracle(inp, t, form=form).active.any(0))
    zero = on[::3]
    assert len(zero) >= 3
    nan = np.uint16(0x7FC0) if wdt == BF16 else np.float32(np.nan)
    inp.w_up = inp.w_up.copy()
    inp.w_down_t = inp.w_down_t.copy()
    inp.w_up[zero] = 0
    inp.w_down_t[zero] = nan
    y, idx, act, _ = gu.run_gpu_ex(gu.DevInputs(inp), t, form)
    res = gu.run_oracle(inp, t, form=form)
    assert np.isfinite(res.y).all()
    gu.check_parity(res, y, idx, act, t, wdt, what=f"s_gated {shape}")


# ---------------------------------------------------------------- the fixed matrices of the LoPA ablation
# (appendix on the ablation of W1's design: the repeated diagonal, its negative, the tiled identity)
@pytest.mark.parametrize("kind", ["diagonal", "minus_diagonal", "tiled"])
@pytest.mark.parametrize("T,d,d_ff,r", [(1, 264, 1000, 40), (1, 4096, 14336, 512), (4, 264, 1000, 40),
                                        (20, 264, 1000, 40)], ids=lambda v: str(v))
def test_fixed_matrix_variants(gu, kind, T, d, d_ff, r):
    inp = wl.make_inputs(206, T, d, d_ff, r=r, wdt=BF16)
    if kind == "tiled":
        g_idx, g_sign = wl.g_tiled_identity(d, d_ff)
    else:
        g_idx, g_sign = wl.g_repeated_diagonal(d, d_ff, -1 if kind == "minus_diagonal" else 1)
    fi = wl.FormInputs(g_idx=g_idx, g_sign=g_sign, rms_gain=np.ones(r, np.float32))
    form = gu.Form(act=1, silu_up=True, form=fi, use_g=True)
    t = 1.2816 * S2
    y, idx, act, _ = gu.run_gpu_ex(gu.DevInputs(inp), t, form)
    res = gu.run_oracle(inp, t, form=form)
    fig = gu.check_parity(res, y, idx, act, t, BF16, what=f"{kind} T={T}", act_value=form.act_value)
    assert 0 < fig["n_union"] < d_ff


def _random_form_cases(n=24, seed=2028):
    """Seeded shapes and option sets of the full form across the dispatch paths (single
    token, element-wise, matrix-core batches of one to four token tiles, several passes)."""
    rng = np.random.default_rng(seed)
    flag_sets = [ACT, ALL, G_ONLY, NORM_ONLY, dict(act=1), dict(silu_up=True), dict(use_g=True, act=1),
                 dict(rms_norm=True, use_gain=True, silu_up=True)]
    cases = []
    while len(cases) < n:
        i = len(cases)
        T = int(rng.choice([1, 1, 1, 2, 3, 4, 7, 16, 17, 40, 64, 70]))
        d = int(rng.choice([64, 136, 264, 1032, 4096, 100, 250]))
        d_ff = int(rng.integers(5, 4000))
        r = int(rng.choice([0, 16, 40, 128, 520, 36]))
        wdt = BF16 if rng.random() < 0.75 else F32
        flags = flag_sets[int(rng.integers(len(flag_sets)))]
        if r == 0:  # G and the norm are LoPA's
            flags = {k: v for k, v in flags.items() if k in ("act", "silu_up")} or dict(act=1)
        if T * d * (d_ff + r) > 2e8:
            continue
        t = 1.2816 * (S2 if flags.get("use_g") else 1.0)
        tag = f"frand{i}_T{T}_d{d}_dff{d_ff}_r{r}_{'bf16' if wdt == BF16 else 'f32'}_" + "+".join(sorted(flags))
        cases.append((tag, T, d, d_ff, r, wdt, t, flags))
    return cases


FRANDOM = _random_form_cases()


@pytest.mark.parametrize("case", FRANDOM, ids=[c[0] for c in FRANDOM])
def test_full_form_random_shapes(gu, case):
    name, T, d, d_ff, r, wdt, t, flags = case
    inp = wl.make_inputs(206, T, d, d_ff, r=r, wdt=wdt)
    form = _form(gu, inp, flags)
    y, idx, act, _ = gu.run_gpu_ex(gu.DevInputs(inp), t, form)
    res = gu.run_oracle(inp, t, form=form)
    gu.check_parity(res, y, idx, act, t, wdt, what=name, act_value=form.act_value)
