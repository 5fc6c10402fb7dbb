"""Caller-given budget per timestep (approx_lstm_run_schedule) and the
online launch's handling of K_t = 0 steps.

A scheduled run is the online (anytime) launch with K_t read from the
caller's schedule instead of the device clock, so the schedule can put K_t = 0
steps right before K_t > 0 steps, and runs of K_t = 0 steps, on purpose.
Every run must equal the oracle's replay of the schedule (Eq. (1) with K_t
terms per gate at timestep t, then the Sec. II cell update) on the library's
exported terms, to the fp32 bar.  The shapes are chosen, and checked with
approx_lstm_plan, so that the P_x of later timesteps are not all resident in
LDS (each timestep's slot is fetched during the one before it) on the tagged
and on the bulk h exchange, and on a single workgroup."""

import numpy as np
import pytest
import torch

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import exported_factors, prep, rel_err, run_gpu, say

pytestmark = pytest.mark.gpu
TOL = 1e-4


def schedule(T, kmax, seed):
    """K_t in [0, kmax]: runs of zeros of length 1..5 between positive
    budgets (the full rank among them), starting and ending anywhere."""
    rng = np.random.default_rng(seed)
    ks = []
    while len(ks) < T:
        ks += [0] * int(rng.integers(1, 6))
        ks += [int(v) for v in rng.choice([1, 2, kmax // 2, kmax], size=int(rng.integers(1, 4)))]
    ks = ks[:T]
    ks[1] = kmax
    return np.array(ks, np.int32)


def run_sched(m, w, ks, h0=None, c0=None):
    x = torch.from_numpy(w.x).cuda()
    h = torch.full((w.T, w.B, w.H), float("nan"), device="cuda")
    c = torch.full((w.B, w.H), float("nan"), device="cuda")
    h0t = None if h0 is None else torch.from_numpy(h0).cuda()
    c0t = None if c0 is None else torch.from_numpy(c0).cuda()
    B.approx_lstm_run_schedule(m, x, ks, h, h0t, c0t, c)
    B.approx_lstm_check(m)
    torch.cuda.synchronize()
    return h.cpu().numpy(), c.cpu().numpy()


def check(m, w, ks, h, c, h0=None, c0=None):
    assert np.any((ks[:-1] == 0) & (ks[1:] > 0)), "schedule must step from K_t = 0 to K_t > 0"
    ho, co = oracle.run_schedule(exported_factors(m), w.b, w.x, [int(v) for v in ks], h0, c0)
    e = rel_err(h, ho)
    ec = float(np.abs(c - co).max() / max(np.abs(co).max(), 1e-6))
    say("  rel err h", e, "c", ec)
    assert e < TOL and ec < TOL, (e, ec)


def test_schedule_tagged_exchange_px_streamed():
    """Two workgroups (tagged h words), P_x fetched one timestep ahead."""
    w = synth.make(64, 32, 600, 1, index=44, xkind="normal")
    m = prep(w, 32, 0.5)
    B.approx_lstm_set_launch(m, 2, 0)
    plan = B.approx_lstm_plan(m, w.T, 1, online=1)
    say("schedule, tiny shape, T=600, 2 workgroups:", plan)
    assert plan["blocks"] == 2 and plan["px_all"] == 0 and plan["bulk_h"] == 0, plan
    ks = schedule(w.T, 32, 1)
    h, c = run_sched(m, w, ks)
    check(m, w, ks, h, c)


def test_schedule_bulk_exchange_px_streamed():
    """Eight sequences at H = 512 on 8 workgroups: bulk h exchange, all
    (level, sequence) pairs in one phase-B pass, P_x fetched one ahead."""
    w = synth.make(512, 512, 48, 8, index=43, xkind="relu")
    say("prepare D=512 H=512 B=8 p=0.75 rank 128")
    m = prep(w, 128, 0.75)
    B.approx_lstm_set_launch(m, 8, 0)
    plan = B.approx_lstm_plan(m, w.T, 8, online=1)
    say("schedule, D=512 H=512 B=8 T=48, 8 workgroups:", plan)
    assert plan["px_all"] == 0 and plan["bulk_h"] == 1 and plan["allpairs"] == 1, plan
    ks = schedule(w.T, 128, 2)
    h, c = run_sched(m, w, ks)
    check(m, w, ks, h, c)


def test_schedule_single_workgroup_px_streamed_with_initial_state():
    w = synth.make(64, 32, 300, 1, index=45, xkind="normal")
    m = prep(w, 32, 0.5)
    B.approx_lstm_set_launch(m, 1, 0)
    plan = B.approx_lstm_plan(m, w.T, 1, online=1)
    say("schedule, tiny shape, T=300, one workgroup:", plan)
    assert plan["blocks"] == 1 and plan["px_all"] == 0, plan
    rng = np.random.default_rng(7)
    h0 = rng.normal(size=(1, 32)).astype(np.float32)
    c0 = rng.normal(size=(1, 32)).astype(np.float32)
    ks = schedule(w.T, 32, 3)
    h, c = run_sched(m, w, ks, h0, c0)
    check(m, w, ks, h, c, h0, c0)


def test_single_workgroup_long_sequence_fixed_levels():
    """A single workgroup with more timesteps than its LDS holds P_x for:
    fixed levels, against the oracle's independent recurrences."""
    w = synth.make(64, 32, 300, 1, index=46, xkind="normal")
    m = prep(w, 32, 0.5)
    B.approx_lstm_set_launch(m, 1, 0)
    levels = [32]
    plan = B.approx_lstm_plan(m, w.T, 1, levels)
    say("one workgroup, T=300, K=32:", plan)
    assert plan["blocks"] == 1 and plan["px_all"] == 0, plan
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(exported_factors(m), w.b, w.x, levels)
    e = rel_err(h, ho)
    say("  rel err", e)
    assert e < TOL, e


def test_schedule_argument_errors():
    w = synth.named("tiny")
    m = prep(w, 8, 0.5)
    x = torch.zeros((4, 1, 64), device="cuda")
    h = torch.zeros((4, 1, 32), device="cuda")
    for bad in ([0, 1, 9, 0], [0, -1, 0, 0]):
        with pytest.raises(B.ApproxLstmError) as ei:
            B.approx_lstm_run_schedule(m, x, np.array(bad, np.int32), h)
        assert ei.value.status == B.ERR_INVALID_ARG
    m16 = prep(w, 8, 0.5, factor_dtype=1)
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_schedule(m16, x, np.zeros(4, np.int32), h)
    assert ei.value.status == B.ERR_UNSUPPORTED
