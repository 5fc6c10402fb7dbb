"""Parity of the HIP run path (through the C ABI) with the float64 oracle.

Error measure: for every (level, timestep, sequence), the max-abs difference
of the H-vector h divided by max(||h_oracle||_inf, 1e-6); the bar is 1e-4
for the fp32 path.  Where the oracle's factor chain is independent of the
library's (tiny workload, and the first steps of the driving workload), the
oracle prepares its own factors; past the chain's agreement horizon (the
residual-SVD-with-pruning chain is numerically chaotic, see
test_library_cpu.py) the oracle runs on the library's exported terms, which
test_library_cpu.py certifies step by step against the oracle.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import exported_factors, prep, rel_err, run_gpu, say

pytestmark = pytest.mark.gpu
TOL = 1e-4


# ------------------------------------------------------------------ tiny
@pytest.mark.parametrize("G", [4, 1])
@pytest.mark.parametrize("p", [0.0, 0.5])
def test_tiny_every_level_matches_oracle(G, p):
    w = synth.named("tiny")
    levels = [0, 1, 4, 16, 96]
    say("tiny", "G", G, "p", p, "levels", levels)
    m = prep(w, 96, p, G)
    f = oracle.prepare(w.W, 32, 96, oracle.nz_from_ratio(96, p), groups=G)
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(f, w.b, w.x, levels)
    for j, K in enumerate(levels):
        assert rel_err(h[j], ho[j]) < TOL, (K, rel_err(h[j], ho[j]))
    if p == 0.0:
        he, _ = oracle.exact_lstm(w.W, w.b, w.x)
        assert rel_err(h[-1], he) < TOL          # full rank, no pruning: the exact LSTM


def test_tiny_batch_with_initial_state_and_final_cell():
    w = synth.make(64, 32, 6, 3, index=11, xkind="normal")
    rng = np.random.default_rng(5)
    h0 = rng.normal(size=(3, 32)).astype(np.float32)
    c0 = rng.normal(size=(3, 32)).astype(np.float32)
    levels = [0, 7, 96]
    say("tiny batch 3 with h0/c0", levels)
    m = prep(w, 96, 0.5)
    f = oracle.prepare(w.W, 32, 96, 48)
    h, c = run_gpu(m, w.x, levels, h0, c0, want_c=True)
    ho, co = oracle.run(f, w.b, w.x, levels, h0, c0)
    assert rel_err(h, ho) < TOL
    assert np.abs(c - co).max() < 1e-4 * max(1.0, np.abs(co).max())


@pytest.mark.parametrize("G", [4, 1])
def test_ragged_shapes_and_launch_widths(G):
    """D, H not multiples of anything; hidden units split unevenly over the
    workgroups; K = 0, partial and full; results must not depend on the
    number of workgroups (every sum has a fixed order)."""
    w = synth.make(50, 37, 5, 2, index=12, xkind="relu")
    rank = 20
    levels = [0, 3, rank]
    say("ragged D=50 H=37 G", G)
    m = prep(w, rank, 0.6, G)
    f = oracle.prepare(w.W, 37, rank, oracle.nz_from_ratio(87, 0.6), groups=G)
    ref = None
    for P, coop in ((0, 0), (1, 0), (5, 0), (16, 1), (37, 0), (64, 0)):
        say("  blocks", P, "cooperative", coop)
        B.approx_lstm_set_launch(m, P, coop)
        h, _ = run_gpu(m, w.x, levels)
        ho, _ = oracle.run(f, w.b, w.x, levels)
        assert rel_err(h, ho) < TOL, P
        if ref is None:
            ref = h
        else:
            assert np.array_equal(h, ref), P


def test_zero_length_sequence_and_bad_levels():
    w = synth.named("tiny")
    m = prep(w, 8, 0.5)
    say("T=0 and argument errors")
    x = torch.zeros((0, 1, 64), device="cuda")
    h = torch.zeros((1, 0, 1, 32), device="cuda")
    assert B.approx_lstm_run(m, x, [4], h) == B.OK
    xt = torch.zeros((2, 1, 64), device="cuda")
    ht = torch.zeros((1, 2, 1, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run(m, xt, [9], ht)
    assert ei.value.status == B.ERR_INVALID_ARG
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run(m, xt, [-1], ht)
    assert ei.value.status == B.ERR_INVALID_ARG
    h17 = torch.zeros((17, 2, 1, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run(m, xt, [1] * 17, h17)
    assert ei.value.status == B.ERR_UNSUPPORTED


# --------------------------------------------------------------- driving
@pytest.fixture(scope="module")
def driving():
    return synth.named("driving")


@pytest.fixture(scope="module")
def driving_p75(driving):
    say("prepare driving p=0.75 rank 512")
    return prep(driving, 512, 0.75)


def test_driving_early_levels_match_independent_oracle(driving, driving_p75):
    """K <= 24 lies inside the chain-agreement horizon: the oracle prepares
    its own factors."""
    levels = [1, 2, 8, 24]
    say("driving p=0.75 levels", levels, "vs oracle-prepared factors")
    f = oracle.prepare(driving.W, 512, 24, 640)
    h, _ = run_gpu(driving_p75, driving.x, levels)
    ho, _ = oracle.run(f, driving.b, driving.x, levels)
    for j, K in enumerate(levels):
        assert rel_err(h[j], ho[j]) < TOL, (K, rel_err(h[j], ho[j]))


def test_driving_all_budgets_match_oracle_on_exported_terms(driving, driving_p75):
    levels = [32, 64, 128, 256, 512]
    say("driving p=0.75 levels", levels, "vs oracle on exported terms")
    f = exported_factors(driving_p75)
    h, _ = run_gpu(driving_p75, driving.x, levels)
    ho, _ = oracle.run(f, driving.b, driving.x, levels)
    for j, K in enumerate(levels):
        assert rel_err(h[j], ho[j]) < TOL, (K, rel_err(h[j], ho[j]))


@pytest.fixture(scope="module", params=[0.5, 0.9], ids=["p50", "p90"])
def driving_other(request, driving):
    p = request.param
    say(f"prepare driving p={p} rank 512")
    return p, prep(driving, 512, p)


def test_driving_other_ratios_early_levels_match_independent_oracle(driving, driving_other):
    """The driving workload's other pruning ratios (NZ = 1280 at 50%, 256 at
    90%): budgets inside the chain-agreement horizon (24 steps at 50%, 16 at
    90%) against factors the oracle prepares itself."""
    p, m = driving_other
    nz = oracle.nz_from_ratio(2560, p)
    levels = [1, 2, 4, 8, 16, 24] if p < 0.9 else [1, 2, 4, 8, 16]
    say(f"driving p={p} (NZ={nz}) levels", levels, "vs oracle-prepared factors")
    f = oracle.prepare(driving.W, 512, max(levels), nz)
    h, _ = run_gpu(m, driving.x, levels)
    ho, _ = oracle.run(f, driving.b, driving.x, levels)
    for j, K in enumerate(levels):
        e = rel_err(h[j], ho[j])
        say("  K", K, "rel err", e)
        assert e < TOL, (K, e)


def test_driving_other_ratios_all_budgets_on_exported_terms(driving, driving_other):
    p, m = driving_other
    levels = [32, 64, 128, 256, 512]
    say(f"driving p={p} levels", levels, "vs oracle on exported terms")
    f = exported_factors(m)
    h, _ = run_gpu(m, driving.x, levels)
    ho, _ = oracle.run(f, driving.b, driving.x, levels)
    for j, K in enumerate(levels):
        e = rel_err(h[j], ho[j])
        say("  K", K, "rel err", e)
        assert e < TOL, (K, e)
    # each budget alone: the bench's single-level launch shape
    for K in (64, 512):
        alone, _ = run_gpu(m, driving.x, [K])
        assert rel_err(alone[0], ho[levels.index(K)]) < TOL, K


def test_driving_levels_are_bitwise_independent(driving, driving_p75):
    say("driving level independence")
    together, _ = run_gpu(driving_p75, driving.x, [512, 1, 64])
    for j, K in enumerate([512, 1, 64]):
        alone, _ = run_gpu(driving_p75, driving.x, [K])
        assert np.array_equal(together[j], alone[0]), K


def test_bulk_and_tagged_h_exchange_agree_bitwise(driving, driving_p75):
    """Five levels of the driving workload exchange h in bulk (5 x 512 values
    per timestep: flag words and coherent 16-byte loads); one level exchanges
    tagged words.  The values exchanged are the same, so every level must
    match its single-level run bit for bit (and the oracle)."""
    levels = [64, 64, 512, 8, 64]
    say("driving: bulk h exchange (5 levels) vs tagged (1 level)")
    together, _ = run_gpu(driving_p75, driving.x, levels)
    for j, K in enumerate(levels):
        alone, _ = run_gpu(driving_p75, driving.x, [K])
        assert np.array_equal(together[j], alone[0]), (j, K)


def test_zero_budget_spreads_over_workgroups():
    """K = 0 (bias-only gates, Eq. (1) with no step) with 20 sequences: the
    workgroups need nothing from each other; any launch width gives the same
    bits, equal to the oracle."""
    w = synth.make(64, 32, 6, 20, index=16, xkind="normal")
    m = prep(w, 8, 0.5)
    f = oracle.prepare(w.W, 32, 8, 48)
    say("K = 0 over 20 sequences, launch widths")
    ref = None
    for P in (0, 1, 3, 8):
        B.approx_lstm_set_launch(m, P, 0)
        h, c = run_gpu(m, w.x, [0], want_c=True)
        ho, co = oracle.run(f, w.b, w.x, [0])
        assert rel_err(h, ho) < TOL, P
        assert np.abs(c - co).max() < TOL * max(1.0, np.abs(co).max())
        if ref is None:
            ref = h
        else:
            assert np.array_equal(h, ref), P


@pytest.mark.parametrize("init", [False, True])
def test_zero_budget_single_pass_equals_general_path(init):
    """A run whose every level has K = 0 takes phase B in one pass over all
    (level, sequence) pairs; a K = 0 level next to a positive budget takes
    the general pass per pair.  Both give the same bits (y is the bias
    alone), with and without an initial state, and equal the oracle."""
    w = synth.make(64, 32, 6, 5, index=17, xkind="normal")
    m = prep(w, 8, 0.5)
    h0 = c0 = None
    if init:
        rng = np.random.default_rng(5)
        h0 = rng.normal(size=(5, 32)).astype(np.float32)
        c0 = rng.normal(size=(5, 32)).astype(np.float32)
    say("K = 0 single pass vs general path, initial state", init)
    hz, cz = run_gpu(m, w.x, [0, 0], h0, c0, want_c=True)
    hm, cm = run_gpu(m, w.x, [0, 5], h0, c0, want_c=True)
    for j in range(2):
        assert np.array_equal(hz[j], hm[0]), j
        assert np.array_equal(cz[j], cm[0]), j
    ho, co = oracle.run(oracle.prepare(w.W, 32, 8, 48), w.b, w.x, [0], h0, c0)
    assert rel_err(hz[0], ho[0]) < TOL
    assert np.abs(cz[0] - co[0]).max() < TOL * max(1.0, np.abs(co[0]).max())


def test_driving_full_rank_without_pruning_is_the_exact_lstm(driving):
    say("driving p=0 rank 512 vs exact LSTM")
    m = prep(driving, 512, 0.0)
    h, _ = run_gpu(m, driving.x, [512])
    he, _ = oracle.exact_lstm(driving.W, driving.b, driving.x)
    assert rel_err(h[0], he) < TOL


# ----------------------------------------------------------------- stack
def oracle_stack(factors, biases, x, levels):
    """Layer-by-layer oracle: layer l at level j reads layer l-1's h at level j."""
    out = []
    for lv in levels:
        inp = x
        for f, b, K in zip(factors, biases, lv):
            hs, _ = oracle.run(f, b, inp, [K])
            inp = hs[0]
        out.append(inp)
    return np.stack(out)


@pytest.mark.parametrize("independent", [True, False])
def test_stack_matches_layerwise_oracle(independent):
    """Two stacked layers (the stacked workload at a quarter of its sizes:
    D=1024 -> H=256 -> H=256, T=8, 75% pruning).  Per-layer budgets; with
    independent=True the oracle prepares its own factors (K inside the chain
    agreement horizon), else it runs on the library's exported terms."""
    w = synth.make(1024, 256, 8, 1, index=14, xkind="relu", n_layers=2)
    (W1, b1), (W2, b2) = w.layers
    levels = [(8, 8), (16, 4)] if independent else [(16, 16), (64, 64), (256, 256), (0, 256), (256, 0)]
    rank = 16 if independent else 256
    say("stack 1024->256->256 levels", levels, "independent", independent)
    m1 = B.approx_lstm_prepare(W1[:, :1024], W1[:, 1024:], b1, 1024, 256, rank, prune_ratio=0.75)
    m2 = B.approx_lstm_prepare(W2[:, :256], W2[:, 256:], b2, 256, 256, rank, prune_ratio=0.75)
    if independent:
        f1 = oracle.prepare(W1, 256, rank, oracle.nz_from_ratio(1280, 0.75))
        f2 = oracle.prepare(W2, 256, rank, oracle.nz_from_ratio(512, 0.75))
    else:
        f1, f2 = exported_factors(m1), exported_factors(m2)
    xt = torch.from_numpy(w.x).cuda()
    h = torch.full((len(levels), 8, 1, 256), float("nan"), device="cuda")
    B.approx_lstm_run_stack([m1, m2], xt, levels, h)
    B.approx_lstm_check(m1)
    B.approx_lstm_check(m2)
    torch.cuda.synchronize()
    ho = oracle_stack([f1, f2], [b1, b2], w.x, levels)
    hg = h.cpu().numpy()
    for j, lv in enumerate(levels):
        assert rel_err(hg[j], ho[j]) < TOL, (lv, rel_err(hg[j], ho[j]))


def test_stack_rejects_mismatched_layers():
    w = synth.named("tiny")
    m1 = prep(w, 4, 0.5)                   # D=64, H=32
    m2 = prep(w, 4, 0.5)                   # expects input 64, gets 32
    xt = torch.zeros((2, 1, 64), device="cuda")
    h = torch.zeros((1, 2, 1, 32), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_stack([m1, m2], xt, [(1, 1)], h)
    assert ei.value.status == B.ERR_INVALID_ARG


# -------------------------------------------------------------- deadline
@pytest.fixture(scope="module")
def deadline_small():
    """The deadline workload at a quarter of its sizes: D=512 -> H=512, T=16,
    batch 2, rank 512, 90% pruning."""
    w = synth.make(512, 512, 16, 2, index=15, xkind="relu")
    say("prepare deadline-shaped D=512 H=512 rank 512 p=0.9")
    m = B.approx_lstm_prepare(w.W[:, :512], w.W[:, 512:], w.b, 512, 512, 512, prune_ratio=0.9)
    return w, m


def test_deadline_mode_picks_budget_and_matches_replay(deadline_small):
    """A generous deadline buys every term; tighter deadlines (fractions of
    the full-rank step time) buy no more terms; every output equals the
    progressive LSTM replayed at the achieved budgets."""
    w, m = deadline_small
    f = exported_factors(m)
    xt = torch.from_numpy(w.x).cuda()
    he, _ = oracle.exact_lstm(w.W, w.b, w.x)
    ks, full_us = [], None
    for frac in (None, 0.8, 0.6):
        dl = 1e6 if frac is None else frac * full_us
        say("deadline", dl, "us/step")
        h = torch.full((16, 2, 512), float("nan"), device="cuda")
        try:
            k, us = B.approx_lstm_run_deadline(m, xt, dl, h)
        except B.ApproxLstmError as e:
            assert e.status == B.ERR_DEADLINE_INFEASIBLE and frac is not None
            say("  infeasible:", str(e))
            continue
        torch.cuda.synchronize()
        if frac is None:
            full_us = float(np.median(us))
        assert np.all(k == k[0]) and 0 <= k[0] <= 512
        ks.append(int(k[0]))
        ho, _ = oracle.run_schedule(f, w.b, w.x, list(k))
        assert rel_err(h.cpu().numpy(), ho) < TOL, dl
        say("  K", k[0], "median step us", float(np.median(us)), "max |h - exact|",
            float(np.abs(h.cpu().numpy() - he).max()))
    assert ks[0] == 512
    assert all(a >= b for a, b in zip(ks, ks[1:]))


def test_deadline_infeasible(deadline_small):
    w, m = deadline_small
    xt = torch.from_numpy(w.x).cuda()
    h = torch.zeros((16, 2, 512), device="cuda")
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_run_deadline(m, xt, 1e-3, h)
    assert ei.value.status == B.ERR_DEADLINE_INFEASIBLE


# ------------------------------------------------------- full-size workloads
def test_stack_full_size_matches_oracle_on_exported_terms():
    """The stacked workload at its full size: D=4096 -> H=1024 -> H=1024,
    T=32, batch 1, rank 1024 per layer, 75% pruning, per-layer budgets
    (64, 64), (256, 256), (1024, 1024); every output against the oracle run
    layer by layer on the library's exported terms."""
    w = synth.named("stack")
    (W1, b1), (W2, b2) = w.layers
    levels = [(64, 64), (256, 256), (1024, 1024)]
    say("stack full size: prepare layer 1 (4 gates of 1024 x 5120, rank 1024)")
    m1 = B.approx_lstm_prepare(W1[:, :4096], W1[:, 4096:], b1, 4096, 1024, 1024, prune_ratio=0.75)
    say("stack full size: prepare layer 2 (rank 1024)")
    m2 = B.approx_lstm_prepare(W2[:, :1024], W2[:, 1024:], b2, 1024, 1024, 1024, prune_ratio=0.75)
    say("stack full size: run levels", levels)
    xt = torch.from_numpy(w.x).cuda()
    h = torch.full((len(levels), 32, 1, 1024), float("nan"), device="cuda")
    B.approx_lstm_run_stack([m1, m2], xt, levels, h)
    B.approx_lstm_check(m1)
    B.approx_lstm_check(m2)
    torch.cuda.synchronize()
    say("stack full size: oracle")
    ho = oracle_stack([exported_factors(m1), exported_factors(m2)], [b1, b2], w.x, levels)
    hg = h.cpu().numpy()
    for j, lv in enumerate(levels):
        e = rel_err(hg[j], ho[j])
        say("  levels", lv, "rel err", e)
        assert e < TOL, (lv, e)


def test_deadline_full_shape_reduced_rank():
    """The deadline workload's shapes (D=2048, H=2048, T=64, batch 8, 90%
    pruning) with rank 256 instead of 2048 (the host factorisation at rank
    2048 takes minutes): deadlines 5, 20 and 100 us per timestep; each run
    that is feasible must equal the oracle replayed at the achieved budgets;
    its error against the exact LSTM is reported."""
    w = synth.named("deadline")
    say("deadline shape: prepare rank 256")
    m = B.approx_lstm_prepare(w.W[:, :2048], w.W[:, 2048:], w.b, 2048, 2048, 256, prune_ratio=0.9)
    f = exported_factors(m)
    xt = torch.from_numpy(w.x).cuda()
    say("deadline shape: exact LSTM (oracle)")
    he, _ = oracle.exact_lstm(w.W, w.b, w.x)
    ks = []
    for dl in (5.0, 20.0, 100.0):
        h = torch.full((64, 8, 2048), float("nan"), device="cuda")
        try:
            k, us = B.approx_lstm_run_deadline(m, xt, dl, h)
        except B.ApproxLstmError as e:
            assert e.status == B.ERR_DEADLINE_INFEASIBLE
            say("  deadline", dl, "us: infeasible:", str(e))
            ks.append(-1)
            continue
        torch.cuda.synchronize()
        assert np.all(k == k[0]) and 0 <= k[0] <= 256
        ks.append(int(k[0]))
        ho, _ = oracle.run_schedule(f, w.b, w.x, list(k))
        hg = h.cpu().numpy()
        e = rel_err(hg, ho)
        say("  deadline", dl, "us: K", int(k[0]), "median step us", float(np.median(us)),
            "rel err vs oracle", e, "max |h - exact| / max |exact|",
            float(np.abs(hg - he).max() / np.abs(he).max()))
        assert e < TOL, dl
    assert ks == sorted(ks) and ks[-1] == 256


# ---------------------------------------------------------- paper shape
@pytest.fixture(scope="module")
def paper():
    return synth.named("paper")


@pytest.mark.parametrize("nz", [4160, 130, 32])
def test_paper_shape_matches_oracle(paper, nz):
    """The paper's model shape (Sec. VI-A: D=8256, H=64, T=100) with
    decaying-spectrum weights, at the three non-zero counts of its error
    curves: budgets up to 128 terms per gate (twice the gate's 64 rows; the
    pruned terms keep refining past the rank of the matrix) against the
    oracle on the exported terms, and the first budgets against the oracle's
    own factors."""
    w = paper
    say("paper shape nz", nz, ": prepare rank 128")
    m = B.approx_lstm_prepare(w.W[:, :w.D], w.W[:, w.D:], w.b, w.D, w.H, 128, nz=nz, groups=4)
    levels = [0, 1, 4, 16, 64, 128]
    h, _ = run_gpu(m, w.x, levels)
    ho, _ = oracle.run(exported_factors(m), w.b, w.x, levels)
    for j, K in enumerate(levels):
        e = rel_err(h[j], ho[j])
        say("  K", K, "rel err (exported terms)", e)
        assert e < TOL, (K, e)
    f = oracle.prepare(w.W, w.H, 4, nz)
    ho, _ = oracle.run(f, w.b, w.x, [1, 4])
    for j, K in enumerate([1, 4]):
        e = rel_err(h[1 + j], ho[j])
        say("  K", K, "rel err (oracle factors)", e)
        assert e < TOL, (K, e)

