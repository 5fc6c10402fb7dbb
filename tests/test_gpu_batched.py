"""Parity of the batched bf16 MFMA path (factor_dtype 1) with the float64 oracle.

The batched configuration stores u and the v values in bf16 and multiplies
bf16 operands with fp32 accumulation; the oracle runs the same arithmetic
definition in float64 (``operand_round='bf16'``: x~ and z rounded to bf16
before the products, factor values rounded fp64 -> fp32 -> bf16).  Error
measure as for the fp32 path (max-abs over the H-vector divided by the
oracle's max-abs); the bar for the bf16 configuration is 2e-2.  Masks are
decided in fp64 before any rounding, so they must equal the oracle's bit for
bit wherever the factor chains agree.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import exported_factors, prep, rel_err, run_gpu, say

pytestmark = pytest.mark.gpu
TOL = 2e-2


def prep16(w, rank, p, groups=4, flags=0):
    return prep(w, rank, p, groups, flags, factor_dtype=1)


def check_levels(h, ho, levels, tol=TOL):
    for j, K in enumerate(levels):
        e = rel_err(h[j], ho[j])
        say("  K", K, "rel err", e)
        assert e < tol, (K, e)


# ------------------------------------------------------------------ small
@pytest.mark.parametrize("G", [4, 1])
def test_batched_tiny_every_level_matches_oracle(G):
    """The tiny model's weights, 5 sequences (one padded 64-wide tile), every
    level of the tiny workload, factors prepared independently by the oracle."""
    w = synth.make(64, 32, 8, 5, index=21, xkind="normal")
    levels = [0, 1, 4, 16, 96]
    say("batched tiny B=5 G", G, "levels", levels)
    m = prep16(w, 96, 0.5, G)
    f = oracle.prepare(w.W, 32, 96, 48, groups=G)
    lib = exported_factors(m)
    assert np.array_equal(lib.mask, f.mask)                 # masks: fp64 decisions, bit-exact
    fb = f.rounded("bf16")
    assert np.abs(lib.U - fb.U).max() <= 2.0 ** -8 * np.abs(fb.U).max()
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(fb, w.b, w.x, levels, operand_round="bf16")
    check_levels(h, ho, levels)


def test_batched_initial_state_and_final_cell():
    w = synth.make(64, 32, 6, 3, index=22, xkind="normal")
    rng = np.random.default_rng(7)
    h0 = rng.normal(size=(3, 32)).astype(np.float32)
    c0 = rng.normal(size=(3, 32)).astype(np.float32)
    levels = [0, 7, 96]
    say("batched B=3 with h0/c0", levels)
    m = prep16(w, 96, 0.5)
    f = exported_factors(m)
    h, c = run_gpu(m, w.x, levels, h0, c0, want_c=True)
    ho, co = oracle.run(f, w.b, w.x, levels, h0, c0, operand_round="bf16")
    check_levels(h, ho, levels)
    for j in range(len(levels)):
        assert np.abs(c[j] - co[j]).max() < TOL * max(1.0, np.abs(co[j]).max())


@pytest.mark.parametrize("G", [4, 1])
@pytest.mark.parametrize("Bn", [3, 70])
def test_batched_ragged_shapes(G, Bn):
    """D = 50 (not a multiple of 4 or 32: element-wise x loads and a padded
    contraction), H = 20 (padded to 32), rank 70 (padded to 96), 3 or 70
    sequences (one or two 64-wide tiles)."""
    w = synth.make(50, 20, 5, Bn, index=23, xkind="relu")
    levels = [0, 5, 33, 70]
    say("batched ragged D=50 H=20 B", Bn, "G", G)
    m = prep16(w, 70, 0.5, G)
    f = exported_factors(m)
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(f, w.b, w.x, levels, operand_round="bf16")
    check_levels(h, ho, levels)


def test_batched_unaligned_input_rows():
    """x starting 4 bytes into its buffer: the x loads take the element-wise
    path; the results must be bitwise those of the aligned run."""
    w = synth.make(64, 32, 4, 9, index=24, xkind="relu")
    levels = [3, 40]
    say("batched unaligned x")
    m = prep16(w, 40, 0.5)
    h_al, _ = run_gpu(m, w.x, levels)
    h_un, _ = run_gpu(m, w.x, levels, x_offset=1)
    assert np.array_equal(h_al, h_un)


def test_batched_errors():
    w = synth.make(64, 32, 2, 2, index=25, xkind="relu")
    m = prep16(w, 8, 0.5)
    say("batched argument errors")
    xt = torch.zeros((2, 2, 64), device="cuda")
    h = torch.zeros((1, 2, 2, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run(m, xt, [9], h)
    assert ei.value.status == B.ERR_INVALID_ARG
    hd = torch.zeros((2, 2, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_deadline(m, xt, 100.0, hd)
    assert ei.value.status == B.ERR_UNSUPPORTED
    assert B.approx_lstm_run(m, torch.zeros((0, 2, 64), device="cuda"), [4],
                             torch.zeros((1, 0, 2, 32), device="cuda")) == B.OK


# ------------------------------------------------- batched workload, 1/4 size
@pytest.fixture(scope="module")
def quarter():
    """The batched workload at a quarter of its sizes: D=512, H=128, T=16,
    64 sequences, rank 128, 75% pruning."""
    w = synth.make(512, 128, 16, 64, index=26, xkind="relu")
    say("prepare batched quarter size, rank 128 p=0.75 bf16")
    return w, prep16(w, 128, 0.75)


def test_batched_quarter_early_levels_match_independent_oracle(quarter):
    w, m = quarter
    levels = [1, 4, 12]
    say("batched quarter levels", levels, "vs oracle-prepared factors")
    f = oracle.prepare(w.W, 128, 12, oracle.nz_from_ratio(640, 0.75))
    lib = exported_factors(m)
    assert np.array_equal(lib.mask[:, :12], f.mask)
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(f.rounded("bf16"), w.b, w.x, levels, operand_round="bf16")
    check_levels(h, ho, levels)


def test_batched_quarter_all_levels_on_exported_terms(quarter):
    w, m = quarter
    levels = [0, 32, 64, 128]
    say("batched quarter levels", levels, "vs oracle on exported terms")
    f = exported_factors(m)
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(f, w.b, w.x, levels, operand_round="bf16")
    check_levels(h, ho, levels)


def test_batched_quarter_levels_bitwise_independent(quarter):
    w, m = quarter
    say("batched quarter level independence")
    together, _ = run_gpu(m, w.x, [128, 5, 64])
    for j, K in enumerate([128, 5, 64]):
        alone, _ = run_gpu(m, w.x, [K])
        assert np.array_equal(together[j], alone[0]), K


# ------------------------------------------------- batched workload, full size
@pytest.fixture(scope="module")
def full():
    w = synth.named("batched")
    say("prepare batched workload D=2048 H=512 B=256 rank 512 p=0.75 bf16")
    return w, prep16(w, 512, 0.75)


def test_batched_full_size_every_sequence(full):
    """Every level of the batched workload at its full size, in the launch
    configuration the benchmark times; the oracle checks all 256 sequences
    (all 16 cohorts of the persistent launch)."""
    w, m = full
    levels = [32, 128, 512]
    say("batched full size levels", levels)
    f = exported_factors(m)
    h, _ = run_gpu(m, w.x, levels)
    assert np.isfinite(h).all()
    say("  oracle, 256 sequences")
    ho, _ = oracle.run(f, w.b, w.x, levels, operand_round="bf16")
    check_levels(h, ho, levels)
    pick = np.arange(256)
    # the per-timestep kernel pair at the same size (the persistent launch is the default)
    try:
        B.approx_lstm_set_batched_path(m, 0)
        hp, _ = run_gpu(m, w.x, levels)
    finally:
        B.approx_lstm_set_batched_path(m, 1)
    say("  per-timestep kernels")
    check_levels(hp[:, :, pick], ho, levels)


# ------------------------------------------- persistent vs per-timestep kernels
def test_batched_persistent_and_per_timestep_paths_agree(quarter):
    """The quarter-size workload through the persistent recurrence (cohorts of
    16 sequences over 4 workgroups each, z and h exchanged through device
    memory) and through the per-timestep kernel pair: both within the bar of
    the oracle on the exported terms, and close to each other (they differ
    only in the fp32 summation order of the two products)."""
    w, m = quarter
    levels = [0, 9, 64, 128]
    say("batched quarter: persistent vs per-timestep kernels", levels)
    f = exported_factors(m)
    ho, _ = oracle.run(f, w.b, w.x, levels, operand_round="bf16")
    try:
        B.approx_lstm_set_batched_path(m, 0)
        h_pair, _ = run_gpu(m, w.x, levels)
    finally:
        B.approx_lstm_set_batched_path(m, 1)
    check_levels(h_pair, ho, levels)
    runs = {}
    for mode in (1, 2, 3):   # automatic, z as tagged words, z behind flags
        try:
            B.approx_lstm_set_batched_path(m, mode)
            runs[mode], _ = run_gpu(m, w.x, levels)
        finally:
            B.approx_lstm_set_batched_path(m, 1)
        say("  persistent mode", mode)
        check_levels(runs[mode], ho, levels)
        for j in range(len(levels)):
            assert rel_err(runs[mode][j], h_pair[j]) < TOL
    # the z exchange's form changes no arithmetic
    assert np.array_equal(runs[2], runs[3])
    assert np.array_equal(runs[1], runs[2])


@pytest.mark.parametrize("blocks", [4, 8])
def test_batched_persistent_cohorts_in_turn(quarter, blocks):
    """4 cohorts of 16 sequences on one or two cohorts' worth of workgroups:
    each workgroup runs several cohorts in turn, reusing the exchange buffers
    with fresh tags; bitwise equal to the run with every cohort in flight."""
    w, m = quarter
    levels = [0, 40, 128]
    say("batched quarter persistent, workgroup cap", blocks)
    wide, _ = run_gpu(m, w.x, levels)
    try:
        B.approx_lstm_set_launch(m, blocks)
        narrow, _ = run_gpu(m, w.x, levels)
        again, _ = run_gpu(m, w.x, levels)
    finally:
        B.approx_lstm_set_launch(m, 0)
    assert np.array_equal(wide, narrow)
    assert np.array_equal(wide, again)
    B.approx_lstm_check(m)
