"""The no-allocation entry point (ffn_sparse_forward_noalloc) against ffn_sparse_forward and
the oracle: the same call with the library's own per-GPU workspace.  Two calls in a row,
the second with a smaller input, so the second runs on the first one's leftover workspace."""
import numpy as np
import pytest

from paper_2609_31975_amd import workloads as wl

pytestmark = pytest.mark.gpu

BF16, F32 = wl.BF16, wl.F32


@pytest.fixture(scope="module")
def gu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from tests import gpu_util
    return gpu_util


def _both(gu, inp, t):
    """(y of the no-allocation call, y of ffn_sparse_forward, its active set)."""
    import torch
    from paper_2609_31975_amd import ffn
    dev = gu.DevInputs(inp)
    T, d = inp.x.shape
    y = torch.full((T, d), float("nan"), dtype=torch.float32, device="cuda")
    ffn.ffn_sparse_forward_noalloc(dev.x, dev.w_gate, dev.w_up, dev.w_down_t, t, y)
    torch.cuda.synchronize()
    y_ref, idx, act, _ = gu.run_gpu(dev, t)
    return y.cpu().numpy(), y_ref, idx, act


@pytest.mark.parametrize("first,second", [((4, 4096, 14336, BF16), (1, 1024, 3000, BF16)),
                                          ((1, 8192, 28672, BF16), (1, 264, 1000, F32)),
                                          ((16, 1032, 5000, BF16), (3, 264, 1000, BF16))],
                         ids=["T4_8b_then_T1", "T1_70b_then_f32", "T16_then_T3"])
def test_noalloc_matches_the_workspace_call(gu, first, second):
    t = 1.2816
    for k, (T, d, d_ff, wdt) in enumerate((first, second)):
        inp = wl.make_inputs(300 + k, T, d, d_ff, r=0, wdt=wdt)
        y, y_ref, idx, act = _both(gu, inp, t)
        res = gu.run_oracle(inp, t)
        assert np.isfinite(y).all(), f"call {k}: y not fully written"
        gu.check_parity(res, y, None, None, t, wdt, what=f"no-alloc call {k}")
        gu.check_parity(res, y_ref, idx, act, t, wdt, what=f"workspace call {k}")
        assert gu.rel_err(y, y_ref) < 1e-6, f"call {k}"   # same kernels; only atomic order differs


def test_noalloc_rejects_a_shape_beyond_its_workspace(gu):
    import torch
    from paper_2609_31975_amd import ffn
    T, d, d_ff = 64, 8192, 28672   # needs about 24 MiB of workspace
    x = torch.zeros((T, d), dtype=torch.float32, device="cuda")
    w = torch.zeros((d_ff, d), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((T, d), dtype=torch.float32, device="cuda")
    with pytest.raises(ffn.FFNError) as e:
        ffn.ffn_sparse_forward_noalloc(x, w, w, w, 1.0, y)
    assert e.value.code == -5
