"""Phase B over every sequence at once with K in tiles (one level, several
sequences, U rows too long for registers or LDS: read from memory).  Each
U entry is read once per timestep and applied to every sequence; per
sequence the sums run in the order of the one-sequence pass, so each
sequence's output equals, bit for bit, the same sequence run alone through
the general kernel at the same launch width.  Every run also meets the
oracle on the library's exported terms (fp32 bar; Sec. III Eq. (1) then the
Sec. II cell update)."""

import numpy as np
import pytest

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import exported_factors, prep, rel_err, run_gpu, say

pytestmark = pytest.mark.gpu
TOL = 1e-4
LDS_CAP = 160 * 1024


@pytest.fixture(scope="module")
def wide():
    """H = 1024 (rank up to 1024), D = 256, 8 sequences of 6 steps, 75%
    pruning, factorised on the device."""
    w = synth.make(256, 1024, 6, 8, index=31, xkind="relu", name="wide")
    say("prepare wide H=1024 rank 1024 p=0.75 (device)")
    m = prep(w, 1024, 0.75, flags=B.FLAG_DEVICE_FACTORISE)
    yield w, m
    B.approx_lstm_set_launch(m, 0, 0)


def tiled_launch(m, T, K, Bs=(8, 4, 3, 2), Ps=(128, 96, 80, 160, 192, 256)):
    """The first (sequences, workgroups) whose plan takes the K-tiled phase B."""
    for Bn in Bs:
        for P in Ps:
            B.approx_lstm_set_launch(m, P, 0)
            plan = B.approx_lstm_plan(m, T, Bn, [K])
            if plan["ktile"] > 0 and plan["lds_bytes"] <= LDS_CAP and plan["blocks"] == P:
                return Bn, P, plan
    B.approx_lstm_set_launch(m, 0, 0)
    return None


@pytest.mark.parametrize("K", [1024, 1000, 961])
def test_ktile_equals_single_sequence_runs_and_oracle(wide, K):
    w, m = wide
    T = w.x.shape[0]
    found = tiled_launch(m, T, K)
    assert found is not None, K
    Bn, P, plan = found
    x = np.ascontiguousarray(w.x[:, :Bn])
    say(f"K={K} blocks={P} B={Bn} plan {plan}")
    assert plan["upt"] == 0
    B.approx_lstm_set_recurrence(m, 1)
    try:
        h, c = run_gpu(m, x, [K], want_c=True)
        for b in range(Bn):
            assert B.approx_lstm_plan(m, T, 1, [K])["ktile"] == 0
            hb, cb = run_gpu(m, x[:, b:b + 1], [K], want_c=True)
            assert np.array_equal(h[:, :, b], hb[:, :, 0]), (K, b)
            assert np.array_equal(c[:, b], cb[:, 0]), (K, b)
    finally:
        B.approx_lstm_set_recurrence(m, 0)
        B.approx_lstm_set_launch(m, 0, 0)
    ho, co = oracle.run(exported_factors(m), w.b, x, [K])
    e = rel_err(h, ho)
    say(f"  rel err {e:.2e}")
    assert e < TOL, e
    assert np.abs(c - co).max() <= TOL * max(1.0, np.abs(co).max())


def test_ktile_tile_boundaries(wide):
    """Budgets one past a tile boundary, ending on one, and a partial last
    tile: the tiles' ranges."""
    w, m = wide
    T = w.x.shape[0]
    found = tiled_launch(m, T, 1024)
    assert found is not None
    Bn, P, plan = found
    kt = plan["ktile"]
    x = np.ascontiguousarray(w.x[:, :Bn])
    fac = exported_factors(m)
    try:
        for K in sorted({kt + 1, 2 * kt, 2 * kt + 16, 1024 - 1}):
            if K > 1024:
                continue
            p = B.approx_lstm_plan(m, T, Bn, [K])
            if p["ktile"] == 0:
                continue   # this budget fits the register or LDS path
            h, _ = run_gpu(m, x, [K])
            ho, _ = oracle.run(fac, w.b, x, [K])
            e = rel_err(h, ho)
            say(f"  K={K} ktile {p['ktile']} rel err {e:.2e}")
            assert e < TOL, (K, e)
    finally:
        B.approx_lstm_set_launch(m, 0, 0)
