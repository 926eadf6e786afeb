"""GPU test of the no-allocation entry point tp_backtest_metrics_noalloc
(for callers that cannot allocate device memory): through the C ABI, its
output equals tp_backtest_metrics with a caller workspace bit for bit, on
calls in a row whose second input is smaller, on the shape that needs the
most scratch, and on the one-launch path; the oracle checks the first call;
and no device memory is taken by the calls."""

import numpy as np
import pytest
import torch

import oracle
from gpu_common import say
from paper_2111_05188_amd import tp
from test_gpu_backtest import check_metrics

pytestmark = pytest.mark.gpu

P = 252.0 * 390


def _series(T, E, seed):
    rng = np.random.default_rng(seed)
    v0 = np.full(E, 1e6) * rng.uniform(0.5, 2.0, E)
    v = v0[None] * np.cumprod(1.0 + rng.normal(2e-5, 1e-3, (T, E)), axis=0)
    if E > 2:
        v[T // 3:, 2] = np.nan
    return v0, v


def _both(T, E, seed):
    v0, v = _series(T, E, seed)
    dv0, dv = torch.from_numpy(v0).cuda(), torch.from_numpy(v).cuda()
    ref = tp.backtest_metrics(dv0, dv, P, 0.02)
    out = torch.full((E, 5), 7.0, dtype=torch.float64, device="cuda")
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    tp.backtest_metrics_noalloc(dv0, dv, P, 0.02, out=out)
    torch.cuda.synchronize()
    free1 = torch.cuda.mem_get_info()[0]
    return v0, v, ref.cpu().numpy(), out.cpu().numpy(), free0, free1


def test_noalloc_equals_workspace_version_on_calls_in_a_row():
    cases = [(98280, 16, 1),    # a year of minute bars, three launches, ~2.6 MB scratch
             (4000, 5, 2),      # a smaller input right after: stale scratch contents
             (15, 16320, 3),    # the shape that needs the most scratch (~4.1 MiB)
             (390, 4096, 4),    # one launch, no scratch
             (700, 3, 5)]       # smaller again
    for i, (T, E, seed) in enumerate(cases):
        say(f"[noalloc] call {i}: T={T} E={E}")
        v0, v, ref, got, free0, free1 = _both(T, E, seed)
        assert np.array_equal(got, ref, equal_nan=True), f"call {i} differs from the workspace call"
        if i > 0:
            assert free1 == free0, "the call took device memory"
        if i == 0:
            want = oracle.backtest_metrics(v0, v, P, 0.02)
            check_metrics(got, want, v0, v, P, 0.02)


def test_noalloc_argument_errors():
    x = torch.zeros(4, dtype=torch.float64, device="cuda")
    v = torch.zeros(3, 4, dtype=torch.float64, device="cuda")
    with pytest.raises(tp.TPError) as ei:
        tp.backtest_metrics_noalloc(x, v, 0.0)
    assert ei.value.code == tp.TP_EINVAL
    L = tp.load()
    assert L.tp_backtest_metrics_noalloc(None, v.data_ptr(), 3, 4, 252.0, 0.0, x.data_ptr(),
                                         None) == tp.TP_EINVAL
