"""Online (anytime) budget per timestep: approx_lstm_run_anytime.

The kernel picks K_t on the device from its own clock and the calibrated
step times, so the schedule is not known in advance; the run must equal the
oracle replaying the reported schedule (oracle.run_schedule on the library's
exported terms) to the fp32 bar, on each exchange path of the recurrence
(tagged words, bulk h, a single workgroup)."""

import numpy as np
import pytest
import torch

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import exported_factors, prep, rel_err, say

pytestmark = pytest.mark.gpu
TOL = 1e-4


def anytime(m, w, deadline):
    x = torch.from_numpy(w.x).cuda()
    h = torch.full((w.T, w.B, w.H), float("nan"), device="cuda")
    k, us = B.approx_lstm_run_anytime(m, x, deadline, h)
    return h.cpu().numpy(), k, us


def check_replay(m, w, h, k):
    ho, _ = oracle.run_schedule(exported_factors(m), w.b, w.x, [int(v) for v in k])
    e = rel_err(h, ho)
    say("  schedule", [int(v) for v in k], "rel err", e)
    assert e < TOL, e


@pytest.fixture(scope="module")
def driving_p75():
    w = synth.named("driving")
    say("prepare driving p=0.75 rank 512")
    return w, prep(w, 512, 0.75)


def test_anytime_generous_deadline_takes_every_term(driving_p75):
    w, m = driving_p75
    say("anytime, driving, deadline 1e5 us")
    h, k, us = anytime(m, w, 1e5)
    assert np.all(k == 512), k
    check_replay(m, w, h, k)


def test_anytime_tight_deadlines_replay_exactly(driving_p75):
    """Deadlines between the calibrated step times at K = 1 and K = 512: the
    choice varies over the sequence and the output is the replay of it; the
    sequence as a whole keeps (loosely) to its time budget."""
    w, m = driving_p75
    x = torch.from_numpy(w.x).cuda()
    h = torch.empty((w.T, w.B, w.H), device="cuda")
    # calibrated costs: forced single-budget runs give the range to aim in
    k512, us512 = B.approx_lstm_run_anytime(m, x, 1e5, h)
    lo = float(np.mean(us512))
    for frac in (0.75, 0.9):
        dl = frac * lo
        say("anytime, driving, deadline", round(dl, 3), "us")
        try:
            h, k, us = anytime(m, w, dl)
        except B.ApproxLstmError as e:
            assert e.status == B.ERR_DEADLINE_INFEASIBLE
            say("  infeasible:", str(e))
            continue
        assert set(int(v) for v in k) <= {0} | {2 ** i for i in range(10)}, k
        say("  step us", [round(float(v), 2) for v in us], "mean", float(np.mean(us)))
        assert float(np.sum(us)) <= 1.25 * w.T * dl + 5.0
        check_replay(m, w, h, k)


def test_anytime_infeasible_deadline(driving_p75):
    w, m = driving_p75
    say("anytime, driving, deadline 0.05 us")
    with pytest.raises(B.ApproxLstmError) as ei:
        anytime(m, w, 0.05)
    assert ei.value.status == B.ERR_DEADLINE_INFEASIBLE


def sweep(m, w, label, full):
    """A generous deadline (every term at every step), then deadlines at 97%
    and 90% of that run's mean step time, where the choice must vary."""
    h, k, us = anytime(m, w, 1e5)
    say("anytime,", label, "deadline 1e5 us: mean step", float(np.mean(us)))
    assert np.all(k == full), k
    check_replay(m, w, h, k)
    mixed = False
    for frac in (0.97, 0.9):
        dl = frac * float(np.mean(us))
        say("anytime,", label, "deadline", round(dl, 3), "us")
        try:
            h2, k2, us2 = anytime(m, w, dl)
        except B.ApproxLstmError as e:
            assert e.status == B.ERR_DEADLINE_INFEASIBLE
            continue
        mixed = mixed or len(set(int(v) for v in k2)) > 1
        check_replay(m, w, h2, k2)
    return mixed


def test_anytime_bulk_h_exchange():
    """Eight sequences at H = 512: h (and K_t) travel through the bulk
    exchange."""
    w = synth.make(2048, 512, 12, 8, index=41, xkind="relu")
    say("prepare D=2048 H=512 B=8 p=0.75 rank 128")
    m = prep(w, 128, 0.75)
    sweep(m, w, "bulk path", 128)


def test_anytime_single_workgroup():
    """One workgroup: nothing is exchanged and K_t stays in LDS."""
    w = synth.named("tiny")
    m = prep(w, 32, 0.5)
    B.approx_lstm_set_launch(m, 1, 0)
    sweep(m, w, "one workgroup", 32)


def test_anytime_rejects_bf16_models_and_bad_arguments():
    w = synth.named("tiny")
    say("anytime argument errors")
    m16 = prep(w, 32, 0.5, factor_dtype=1)
    x = torch.zeros((2, 1, 64), device="cuda")
    h = torch.zeros((2, 1, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_anytime(m16, x, 10.0, h)
    assert ei.value.status == B.ERR_UNSUPPORTED
    m = prep(w, 8, 0.5)
    for dl in (0.0, -1.0):
        with pytest.raises(B.ApproxLstmError) as ei:
            B.approx_lstm_run_anytime(m, x, dl, h)
        assert ei.value.status == B.ERR_INVALID_ARG


def test_anytime_with_initial_state():
    """h0 and c0 given: the replay starts from the same state."""
    w = synth.named("tiny")
    m = prep(w, 32, 0.5)
    rng = np.random.default_rng(12)
    h0 = rng.normal(size=(1, 32)).astype(np.float32)
    c0 = rng.normal(size=(1, 32)).astype(np.float32)
    x = torch.from_numpy(w.x).cuda()
    h = torch.full((w.T, 1, 32), float("nan"), device="cuda")
    say("anytime with initial state")
    k, us = B.approx_lstm_run_anytime(m, x, 1e5, h, torch.from_numpy(h0).cuda(), torch.from_numpy(c0).cuda())
    ho, _ = oracle.run_schedule(exported_factors(m), w.b, w.x, [int(v) for v in k], h0, c0)
    assert rel_err(h.cpu().numpy(), ho) < TOL
