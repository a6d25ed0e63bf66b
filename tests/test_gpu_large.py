"""GPU parity on weight matrices around 2 GiB, the most the fast kernels address with 32-bit
byte offsets: just below it the fast kernels run at their largest offsets, past it the calls
take the element-wise kernels, which address rows in 64 bits.

Each large matrix is zero except for K rows spread over its whole address range (the first
rows, rows on both sides of byte 2^31, the last row), which hold a seeded K-row weight set.  A
zero gate row gives h = 0 < t, so those neurons are inactive and their W_up / W_down rows add
nothing: the oracle on the K-row FFN is the exact reference for y, and the active list must be
the active ones of the K rows, at their places in the large matrix.
"""
import numpy as np
import pytest

from paper_2609_31975_amd import workloads as wl

pytestmark = pytest.mark.gpu

T_GATE = 0.3  # zero rows (h = 0) sit 0.3 below it, far outside the 1e-3 band

# name, T, d, d_ff, r, weight format, rows holding weights (ascending)
CASES = [
    # bf16 rows of 16 KB: row 131072 starts at byte 2^31, the matrices hold 2^31 + 128 KB
    ("std_d8192_T1", 1, 8192, 131080, 0, wl.BF16,
     [0, 1, 2, 40000, 65535, 65536, 100000, 131070, 131071, 131072, 131073, 131075, 131078, 131079]),
    ("std_d8192_T3", 3, 8192, 131080, 0, wl.BF16,
     [0, 3, 70000, 131069, 131071, 131072, 131074, 131077, 131079]),
    # fp32 rows of 16 KB likewise
    ("std_f32_d4096_T1", 1, 4096, 131080, 0, wl.F32,
     [0, 1, 65536, 131071, 131072, 131073, 131076, 131079]),
    # just below 2^31 bytes (2^31 - 128 KB): the single-token kernels, the two-workgroup batch
    # kernel and LoPA's single-token kernel with z inside, at their largest row offsets
    ("std_d8192_T1_fast_edge", 1, 8192, 131064, 0, wl.BF16, [0, 1, 65536, 131056, 131060, 131061, 131062, 131063]),
    ("std_d8192_T8_fast_edge", 8, 8192, 131064, 0, wl.BF16, [0, 65536, 131059, 131060, 131062, 131063]),
    ("lopa_d8192_T1_fast_edge", 1, 8192, 131064, 1024, wl.BF16, [0, 2, 98304, 131057, 131061, 131062, 131063]),
    # int8 codes just below 2^31 bytes (8 KB rows, the widest rows of the single-token integer-dot
    # kernels); four tokens take the element-wise batch kernels with codes
    ("i8_d8192_T1_fast_edge", 1, 8192, 262136, 0, wl.I8, [0, 1, 131072, 262128, 262133, 262134, 262135]),
    ("i8_d8192_T4", 4, 8192, 262136, 0, wl.I8, [0, 100000, 262130, 262132, 262134, 262135]),
    # LoPA: B rows of 1032 bf16 (2064 bytes), the largest d_ff the calls take (2^20); row 1040448
    # is the first B row past byte 2^31; W_up / W_down are exactly 2 GiB
    ("lopa_dff2p20_T1", 1, 1024, 1 << 20, 1032, wl.BF16,
     [0, 1, 5000, 524288, 1040447, 1040448, 1040449, 1048000, 1048574, 1048575]),
]


@pytest.fixture(scope="module")
def gu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from tests import gpu_util
    return gpu_util


RUNS = [(c, False) for c in CASES] + [(CASES[0], True)]  # the dense baseline once


@pytest.mark.parametrize("case,dense", RUNS, ids=[c[0] + ("-dense" if dn else "-sparse") for c, dn in RUNS])
def test_matrices_around_2gib(gu, case, dense):
    import torch
    from paper_2609_31975_amd import ffn
    name, T, d, d_ff, r, wdt, rows = case
    K = len(rows)
    assert rows == sorted(set(rows)) and rows[-1] < d_ff
    inp = wl.make_inputs(seed=4242 + len(name), T=T, d=d, d_ff=K, r=r, wdt=wdt)
    where = torch.tensor(rows, dtype=torch.int64, device="cuda")

    tdt = {wl.BF16: torch.bfloat16, wl.F32: torch.float32, wl.I8: torch.int8}[wdt]

    def big(cols, small):
        m = torch.zeros((d_ff, cols), dtype=tdt, device="cuda")
        m[where] = gu.to_dev(small)
        return m

    def big_scale(small):  # one fp32 scale a row; the zero rows' scales are 1
        v = torch.ones(d_ff, dtype=torch.float32, device="cuda")
        v[where] = gu.to_dev(small)
        return v

    print(f"[large] {name} {'dense' if dense else 'sparse'}: d {d} d_ff {d_ff} r {r} T {T}", flush=True)
    x = gu.to_dev(inp.x)
    w_up, w_down_t = big(d, inp.w_up), big(d, inp.w_down_t)
    gate = (gu.to_dev(inp.lopa_a), big(r, inp.lopa_b)) if r else (big(d, inp.w_gate),)
    ws = ffn.alloc_workspace(T, d, d_ff, r)
    y = torch.full((T, d), float("nan"), dtype=torch.float32, device="cuda")
    if wdt == wl.I8:
        assert r == 0 and not dense
        sc = ffn.scales(gate=big_scale(inp.scales["gate"]), up=big_scale(inp.scales["up"]),
                        down=big_scale(inp.scales["down"]))
        ffn.ffn_sparse_forward_q(x, *gate, w_up, w_down_t, sc, T_GATE, None, y, ws)
    else:
        if r:
            fn = ffn.ffn_lopa_dense_forward if dense else ffn.ffn_lopa_sparse_forward
        else:
            fn = ffn.ffn_dense_forward if dense else ffn.ffn_sparse_forward
        fn(x, *gate, w_up, w_down_t, T_GATE, y, ws)
    torch.cuda.synchronize()
    y_gpu = y.cpu().numpy()
    res = gu.run_oracle(inp, T_GATE, dense=dense)
    if dense:
        gu.check_parity(res, y_gpu, None, None, T_GATE, wdt, what=name)
        return
    idx, act = ffn.ffn_active_set(ws, T, d, d_ff, r)
    pos = {row: k for k, row in enumerate(rows)}
    stray = [int(i) for i in idx if int(i) not in pos]
    assert not stray, f"{name}: neurons with zero gate rows listed: {stray[:10]}"
    idx_k = np.array([pos[int(i)] for i in idx], dtype=np.int64)
    out = gu.check_parity(res, y_gpu, idx_k, act, T_GATE, wdt, what=name)
    assert out["n_union"] > 0, f"{name}: no active neuron; the case checks nothing"
