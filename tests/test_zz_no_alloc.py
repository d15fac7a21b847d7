"""The entry point that allocates nothing (baseline_rmsnorm_linear_noalloc), called
through the C ABI, against baseline_rmsnorm_linear with a caller workspace: the same
kernels on the same inputs, so the outputs must be bitwise equal; both are also
checked against the fp64 oracle's standard form (RMSNorm then the product, Sec. 3.1).
Two calls in a row, the second smaller, show that the shared static workspace carries
nothing from one call into the next; the largest input that fits is checked too."""
import numpy as np
import pytest
import torch

import __graft_entry__ as graft
import oracle
from paper_2407_09577_amd import workloads

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def fn():
    graft.ensure_built()
    from paper_2407_09577_amd import flashnorm
    flashnorm.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return flashnorm


def _row_err(got, ref):
    got = got.float().cpu().double().numpy()
    assert np.isfinite(got).all()
    return float(np.max(np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)))


def _both(fn, w, path=0, rows=None):
    a, g = w.a.to(DEV), w.g.to(DEV)
    Wp, _, _ = fn.fold_weights(w.W.to(DEV), None)  # the unfolded packed weight of the unfused chain
    x_ws = torch.empty(w.M, w.K, dtype=w.dtype, device=DEV)
    ld = (w.N + 7) // 8 * 8  # output rows 16-byte aligned
    y_ws = torch.empty(w.M, ld, dtype=w.dtype, device=DEV)[:, :w.N]
    y_na = torch.full((w.M, ld), float("nan"), dtype=w.dtype, device=DEV)[:, :w.N]
    fn.baseline_rmsnorm_linear(a, g, Wp, w.N, w.eps, x_ws=x_ws, out=y_ws, path=path)
    fn.baseline_rmsnorm_linear_noalloc(a, g, Wp, w.N, w.eps, out=y_na, path=path)
    torch.cuda.synchronize()
    ref = oracle.rmsnorm_linear(w.a, w.g, w.W, w.eps, rows=rows)
    return y_ws, y_na, ref


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_noalloc_two_calls_second_smaller(fn, dtype):
    for M, K, N, path in [(1000, 576, 1536, 0), (300, 200, 333, 0), (7, 264, 136, 2)]:
        if dtype == torch.float32 and path == 2:
            path = 0
        w = workloads.make("linear", M, K, N, dtype=dtype, eps=1e-5, seed=M + K, outlier_frac=0.02)
        y_ws, y_na, ref = _both(fn, w, path)
        bits = torch.int16 if dtype == torch.bfloat16 else torch.int32
        assert torch.equal(y_ws.view(bits), y_na.view(bits)), (M, K, N)
        assert _row_err(y_na, ref) <= (2e-2 if dtype == torch.bfloat16 else 1e-5)


def test_noalloc_largest_input_that_fits(fn):
    # 4096 x 4096 bf16 activations fill the 32 MiB array exactly (Llama-7B QKV shape);
    # one more row is refused with FN_ERR_SIZE before anything is launched.
    w = workloads.llama7b_qkv_prefill()
    rows = np.array([0, 1, 255, 256, 2047, 2048, 4094, 4095])
    y_ws, y_na, ref = _both(fn, w, rows=rows)
    assert torch.equal(y_ws.view(torch.int16), y_na.view(torch.int16))
    assert _row_err(y_na[torch.from_numpy(rows).to(DEV)], ref) <= 2e-2
    a = torch.zeros(4097, 4096, dtype=torch.bfloat16, device=DEV)
    Wp = torch.zeros(fn.fold_weights_size(4096, 64), dtype=torch.uint8, device=DEV)
    with pytest.raises(fn.FlashNormError) as e:
        fn.baseline_rmsnorm_linear_noalloc(a, torch.ones(4096, device=DEV), Wp, 64, 1e-6)
    assert e.value.status == -9
