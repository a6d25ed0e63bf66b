"""The parity rule of the GPU tests (tests/gpu_util.check_parity) has teeth: an output built
from the oracle itself passes it, and each planted error a kernel could make is rejected
(CPU only: the "GPU outputs" here are the oracle's, altered by hand)."""
import numpy as np
import pytest

from paper_2609_31975_amd import workloads as wl
from tests import gpu_util as gu

T_GATE = 1.0


def _case(T=3, d=512, d_ff=700, wdt=wl.BF16, seed=611):
    """The oracle's result and the (y, idx, act) a correct kernel would return."""
    inp = wl.make_inputs(seed, T, d, d_ff, wdt=wdt)
    res = gu.run_oracle(inp, T_GATE)
    idx = np.flatnonzero(res.active.any(0)).astype(np.int32)
    t32 = np.float64(np.float32(T_GATE))
    act = np.where(res.active[:, idx], res.h[:, idx] - t32, 0.0).astype(np.float32)
    return res, res.y.astype(np.float32), idx, act


def _outside_band(res, tau):
    """A neuron active for token tau, and one inactive for every token, both clear of the band."""
    far = ~(np.abs(res.h - T_GATE) < gu.BAND).any(0)
    on = np.flatnonzero(res.active[tau] & far)
    off = np.flatnonzero(~res.active.any(0) & far)
    return int(on[len(on) // 2]), int(off[len(off) // 2])


def test_exact_output_passes():
    res, y, idx, act = _case()
    out = gu.check_parity(res, y, idx, act, T_GATE, wl.BF16, what="exact")
    assert out["n_union"] == len(idx) and out["band_flips"] == 0


@pytest.mark.parametrize("wdt", [wl.BF16, wl.F32])
def test_one_column_off_fails(wdt):
    """One column off by 1.5x the tolerance of the largest entry: too small to move the
    per-token norm past its bound at d = 4096, caught by the element-wise bound."""
    res, y, idx, act = _case(T=1, d=4096, d_ff=300, wdt=wdt)
    bad = y.copy()
    j = int(np.argmax(np.abs(res.y[0])))
    bad[0, j] += np.float32(1.5 * gu.TOL[wdt] * np.max(np.abs(res.y[0])))
    assert gu.rel_err(bad[0], res.y[0]) < gu.TOL[wdt]  # the norm alone would pass it
    with pytest.raises(AssertionError, match="max abs error"):
        gu.check_parity(res, bad, idx, act, T_GATE, wdt, what="one column")


def test_scaled_token_fails():
    res, y, idx, act = _case()
    bad = y.copy()
    bad[1] *= np.float32(1.01)
    with pytest.raises(AssertionError, match="relative error"):
        gu.check_parity(res, bad, idx, act, T_GATE, wl.BF16, what="scaled token")


def test_missing_active_neuron_fails():
    res, y, idx, act = _case()
    on, _ = _outside_band(res, 0)
    keep = idx != on
    with pytest.raises(AssertionError, match="active-set mismatch"):
        gu.check_parity(res, y, idx[keep], act[:, keep], T_GATE, wl.BF16, what="missing neuron")


def test_extra_inactive_neuron_fails():
    res, y, idx, act = _case()
    _, off = _outside_band(res, 0)
    idx2 = np.sort(np.append(idx, off)).astype(np.int32)
    act2 = np.zeros((act.shape[0], len(idx2)), np.float32)
    pos = np.searchsorted(idx2, idx)
    act2[:, pos] = act
    act2[0, np.searchsorted(idx2, off)] = 0.5  # listed as active for token 0
    with pytest.raises(AssertionError, match="active-set mismatch"):
        gu.check_parity(res, y, idx2, act2, T_GATE, wl.BF16, what="extra neuron")


def test_listed_but_never_active_fails():
    """A neuron in the list that no token activates (zero activations): the list must be the
    union of the active sets exactly."""
    res, y, idx, act = _case()
    _, off = _outside_band(res, 0)
    idx2 = np.sort(np.append(idx, off)).astype(np.int32)
    act2 = np.zeros((act.shape[0], len(idx2)), np.float32)
    act2[:, np.searchsorted(idx2, idx)] = act
    with pytest.raises(AssertionError, match="union"):
        gu.check_parity(res, y, idx2, act2, T_GATE, wl.BF16, what="listed, inactive")


def test_flip_inside_the_band_passes():
    """A neuron within 1e-3 of the threshold may go either way."""
    inp = wl.make_inputs(612, 1, 256, 4000, wdt=wl.F32)
    res = gu.run_oracle(inp, T_GATE)
    near = np.flatnonzero(np.abs(res.h[0] - T_GATE) < gu.BAND)
    assert near.size, "no neuron in the band for this seed"
    k = int(near[0])
    active = res.active[0].copy()
    active[k] = not active[k]
    idx = np.flatnonzero(active).astype(np.int32)
    act = (res.h[0, idx] - np.float64(np.float32(T_GATE))).astype(np.float32)[None, :]
    if active[k]:  # now listed: its value is h - t, within 1e-3 of 0 either way
        act[0, np.searchsorted(idx, k)] = np.float32(max(res.h[0, k] - T_GATE, 1e-7))
    y = res.y.astype(np.float32)  # the flip moves y by |h - t| |v| |d_i|, far inside the tolerance
    out = gu.check_parity(res, y, idx, act, T_GATE, wl.F32, what="band flip")
    assert out["band_flips"] == 1


def test_wrong_activation_value_fails():
    res, y, idx, act = _case()
    bad = act.copy()
    on, _ = _outside_band(res, 0)
    bad[0, np.searchsorted(idx, on)] += np.float32(1e-3)
    with pytest.raises(AssertionError, match="activation values"):
        gu.check_parity(res, y, idx, bad, T_GATE, wl.BF16, what="activation")


def test_unsorted_list_fails():
    res, y, idx, act = _case()
    with pytest.raises(AssertionError, match="ascending"):
        gu.check_parity(res, y, idx[::-1].copy(), act[:, ::-1].copy(), T_GATE, wl.BF16, what="order")


def test_non_finite_output_fails():
    res, y, idx, act = _case()
    bad = y.copy()
    bad[2, 5] = np.nan
    with pytest.raises(AssertionError, match="non-finite"):
        gu.check_parity(res, bad, idx, act, T_GATE, wl.BF16, what="nan")


def test_nothing_active_needs_exact_zeros():
    inp = wl.make_inputs(613, 2, 128, 200, wdt=wl.F32)
    res = gu.run_oracle(inp, 1e30)
    assert not res.active.any() and not res.y.any()
    empty = np.zeros(0, np.int32)
    gu.check_parity(res, np.zeros((2, 128), np.float32), empty, np.zeros((2, 0), np.float32), 1e30, wl.F32)
    tiny = np.zeros((2, 128), np.float32)
    tiny[1, 3] = 1e-30
    with pytest.raises(AssertionError):
        gu.check_parity(res, tiny, empty, np.zeros((2, 0), np.float32), 1e30, wl.F32, what="not zero")


def test_rebuilt_rule_passes_oracle_activations_and_catches_a_missing_term():
    """check_rebuilt: y formed from the oracle's own activations passes; dropping one listed
    neuron's term, or moving one column by 1e-3 of its value, fails."""
    inp = wl.make_inputs(614, 2, 48, 40, wdt=wl.F32)
    res = gu.run_oracle(inp, 0.5)
    idx = np.flatnonzero(res.active.any(0)).astype(np.int32)
    act = np.where(res.active[:, idx], res.h[:, idx] - np.float64(np.float32(0.5)), 0.0).astype(np.float32)
    y = res.y.astype(np.float32)
    gu.check_rebuilt(inp, y, idx, act, wl.F32, what="exact")
    wu = gu.decode_rows(inp.w_up, wl.F32)[idx]
    wd = gu.decode_rows(inp.w_down_t, wl.F32)[idx]
    k = int(np.flatnonzero(act[0])[0])
    missing = y.copy()
    missing[0] -= np.float32(act[0, k] * (inp.x[0].astype(np.float64) @ wu[k])) * wd[k].astype(np.float32)
    with pytest.raises(AssertionError, match="token 0"):
        gu.check_rebuilt(inp, missing, idx, act, wl.F32, what="missing term")
    col = y.copy()
    j = int(np.argmax(np.abs(y[1])))
    col[1, j] *= np.float32(1.001)
    with pytest.raises(AssertionError, match="token 1"):
        gu.check_rebuilt(inp, col, idx, act, wl.F32, what="one column")
