"""approx_lstm_run_noalloc: the run whose workspace is the library's static
device scratch (for callers that cannot allocate).  Through the C ABI, its
outputs must equal approx_lstm_run's on the same model and inputs (same
kernels: bitwise) and the oracle's to the fp32 bar, on two calls in a row,
the second with a smaller input; sizes beyond the scratch are refused."""

import numpy as np
import pytest
import torch

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import exported_factors, prep, rel_err, say

pytestmark = pytest.mark.gpu
TOL = 1e-4


def both_runs(m, x_np, levels, h0=None, c0=None):
    T, Bn, D = x_np.shape
    H = m.hidden_size
    x = torch.from_numpy(np.ascontiguousarray(x_np)).cuda()
    h0t = None if h0 is None else torch.from_numpy(h0).cuda()
    c0t = None if c0 is None else torch.from_numpy(c0).cuda()
    outs = []
    for fn in (B.approx_lstm_run_noalloc, B.approx_lstm_run):
        h = torch.full((len(levels), T, Bn, H), float("nan"), device="cuda")
        c = torch.full((len(levels), Bn, H), float("nan"), device="cuda")
        fn(m, x, levels, h, h0t, c0t, c)
        B.approx_lstm_check(m)
        torch.cuda.synchronize()
        outs.append((h.cpu().numpy(), c.cpu().numpy()))
    return outs


def check(m, w_b, x_np, levels, h0=None, c0=None):
    (hn, cn), (hr, cr) = both_runs(m, x_np, levels, h0, c0)
    assert np.array_equal(hn, hr) and np.array_equal(cn, cr)
    ho, co = oracle.run(exported_factors(m), w_b, x_np, levels, h0, c0)
    e = rel_err(hn, ho)
    say("  rel err vs oracle", e)
    assert e < TOL, e


def test_noalloc_equals_run_twice_second_smaller():
    """The driving workload (the timed configuration, levels and one level),
    then a smaller input (fewer timesteps and terms) on the same scratch."""
    w = synth.named("driving")
    say("no-alloc: prepare driving p=0.75 rank 512")
    m = prep(w, 512, 0.75)
    say("no-alloc: call 1, driving T=16 levels [512, 8, 64]")
    check(m, w.b, w.x, [512, 8, 64])
    say("no-alloc: call 2, driving T=5 level [32]")
    check(m, w.b, w.x[:5], [32])


def test_noalloc_small_model_after_large_and_bulk_exchange():
    """A second model on the same device reuses the scratch: the tiny model
    with initial state, then eight sequences at H = 512 (bulk h exchange)."""
    w = synth.named("tiny")
    m = prep(w, 32, 0.5)
    rng = np.random.default_rng(5)
    h0 = rng.normal(size=(1, 32)).astype(np.float32)
    c0 = rng.normal(size=(1, 32)).astype(np.float32)
    say("no-alloc: tiny, levels [0, 1, 4, 16, 32], initial state")
    check(m, w.b, w.x, [0, 1, 4, 16, 32], h0, c0)
    wb = synth.make(512, 512, 12, 8, index=43, xkind="relu")
    mb = prep(wb, 128, 0.75)
    say("no-alloc: D=512 H=512 B=8, level [128] (bulk h)")
    check(mb, wb.b, wb.x, [128])
    say("no-alloc: D=512 H=512 B=3 T=4, level [16]")
    check(mb, wb.b, wb.x[:4, :3], [16])


def test_noalloc_refuses_runs_beyond_the_scratch():
    """A run whose x-part projections alone exceed 32 MiB is refused with
    UNSUPPORTED before any device work; so is a bf16 model."""
    w = synth.named("tiny")
    m = prep(w, 32, 0.5)
    T, Bn = 4096, 80   # 4 groups x 32 terms x 4096 x 80 x 4 bytes = 160 MiB of P_x
    x = torch.zeros((T, Bn, 64), device="cuda")
    h = torch.zeros((1, T, Bn, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_noalloc(m, x, [32], h)
    assert ei.value.status == B.ERR_UNSUPPORTED and "scratch" in str(ei.value)
    m16 = prep(w, 8, 0.5, factor_dtype=1)
    x2 = torch.zeros((2, 1, 64), device="cuda")
    h2 = torch.zeros((1, 2, 1, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_noalloc(m16, x2, [4], h2)
    assert ei.value.status == B.ERR_UNSUPPORTED
