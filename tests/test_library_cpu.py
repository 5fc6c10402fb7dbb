"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host float64 factorisation agrees with the oracle (masks bit-exact).

The greedy residual-SVD-with-pruning chain is numerically chaotic on random
Gaussian weights (a 1e-13 change in one singular vector grows about tenfold
every two to three steps), so two correct float64 implementations agree
bit-exactly only on a prefix of the chain.  Beyond it, parity is checked one
step at a time: the oracle takes step n from the residual rebuilt from the
library's own earlier terms, and must produce the same sigma, vectors and mask.
"""

import os
import re

import numpy as np
import pytest

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B
from tests.onestep import check_steps

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "approx_lstm.h")
HOST = B.FLAG_HOST_ONLY | B.FLAG_KEEP_UNPRUNED


def prep(w, rank, nz=0, p=0.0, groups=4, flags=HOST):
    D, H = w.D, w.H
    return B.approx_lstm_prepare(w.W[:, :D], w.W[:, D:], w.b, D, H, rank, nz=nz, prune_ratio=p,
                                 groups=groups, flags=flags)


def test_library_exports_every_declared_function():
    text = open(HEADER).read()
    names = set(re.findall(r"\b(approx_lstm_[a-z0-9_]+)\s*\(", text))
    assert {"approx_lstm_prepare", "approx_lstm_run", "approx_lstm_destroy"} <= names
    for n in sorted(names):
        assert hasattr(B.lib, n), n


@pytest.mark.parametrize("G", [4, 1])
@pytest.mark.parametrize("p", [0.0, 0.5])
def test_tiny_chain_bit_exact_with_oracle(G, p):
    """Tiny workload (D=64, H=32): the whole chain (96 steps) matches."""
    w = synth.named("tiny")
    nz = oracle.nz_from_ratio(96, p)
    m = prep(w, 96, p=p, groups=G)
    f = oracle.prepare(w.W, 32, 96, nz, groups=G)
    info = m.info
    assert info["nz"] == nz and info["eff_rank"] == list(f.eff_rank)
    assert info["unconverged_steps"] == 0 and m.status == B.OK
    for g in range(G):
        lf = B.approx_lstm_get_factors(m, g)
        l64 = B.approx_lstm_get_factors_f64(m, g)
        assert np.array_equal(lf["v_idx"], f.mask[g])                      # masks and order
        np.testing.assert_allclose(l64["sigma"], f.sigma[g], rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(l64["u"], f.U[g], atol=1e-9)
        np.testing.assert_allclose(l64["v"], f.v_full[g], atol=1e-9)
        # the stored fp32 values are the fp64 ones rounded to nearest
        assert np.array_equal(lf["sigma"], l64["sigma"].astype(np.float32))
        assert np.array_equal(lf["u"], l64["u"].astype(np.float32))
        vsel = np.take_along_axis(l64["v"], lf["v_idx"].astype(np.int64), axis=1)
        assert np.array_equal(lf["v_val"], vsel.astype(np.float32))


@pytest.fixture(scope="module")
def driving():
    return synth.named("driving")


@pytest.mark.parametrize("p,steps", [(0.5, 24), (0.75, 24), (0.9, 16)])
def test_driving_chain_prefix_bit_exact(driving, p, steps):
    """Driving-shaped workload (D=2048, H=512): the first steps of every gate
    match the oracle's chain bit-exactly (inside the measured agreement
    horizon, which shrinks as pruning grows: about 40 steps at 75%)."""
    C = 2560
    nz = oracle.nz_from_ratio(C, p)
    m = prep(driving, steps, p=p)
    f = oracle.prepare(driving.W, 512, steps, nz)
    for g in range(4):
        lf = B.approx_lstm_get_factors(m, g)
        assert np.array_equal(lf["v_idx"], f.mask[g]), g
        # sigma drifts apart along the chain (the chaos above) while the masks
        # still agree: at 90% pruning the gap reaches ~1e-7 by step 24
        l64 = B.approx_lstm_get_factors_f64(m, g)
        np.testing.assert_allclose(l64["sigma"], f.sigma[g], rtol=1e-7)


@pytest.fixture(scope="module")
def driving_full_p75(driving):
    return prep(driving, 512, p=0.75)


def test_driving_full_chain_one_step_parity(driving, driving_full_p75):
    """Full rank-512 chain at 75% pruning (the timed workload): at sampled
    steps across the chain, the oracle's own step from the library's residual
    gives the same sigma, u, v and, bit-exactly, the same mask."""
    m = driving_full_p75
    assert m.info["eff_rank"] == [512] * 4 and m.info["unconverged_steps"] == 0
    W = driving.W.astype(np.float64)
    steps = [0, 1, 2, 63, 64, 127, 255, 300, 447, 511]
    for g in range(4):
        lf = B.approx_lstm_get_factors(m, g)
        l64 = B.approx_lstm_get_factors_f64(m, g)
        res = check_steps(W[g * 512:(g + 1) * 512], l64["sigma"], l64["u"], l64["v"],
                          lf["v_idx"].astype(np.int64), 640, steps)
        assert all(s == "exact" for _, s in res), res


def test_driving_full_chain_certificates(driving, driving_full_p75):
    """Residual-energy identity (P2) along the whole exported chain: with
    u^T R = sigma v^T, ||R^(n+1)||_F^2 = ||R^(n)||_F^2 - sigma^2 ||v'||^2, so
    ||W - W~^(K)||_F^2 computed from the terms equals the accumulated sum."""
    m = driving_full_p75
    W = driving.W.astype(np.float64)
    for g in (0, 3):
        Wg = W[g * 512:(g + 1) * 512]
        lf = B.approx_lstm_get_factors(m, g)
        l64 = B.approx_lstm_get_factors_f64(m, g)
        idx = lf["v_idx"].astype(np.int64)
        vp = np.take_along_axis(l64["v"], idx, axis=1)
        R = Wg.copy()
        e0 = np.sum(Wg * Wg)
        acc = e0
        for n in range(512):
            R[:, idx[n]] -= l64["sigma"][n] * np.outer(l64["u"][n], vp[n])
            acc -= l64["sigma"][n] ** 2 * np.sum(vp[n] ** 2)
            if n in (0, 10, 100, 511):
                assert abs(np.sum(R * R) - acc) <= 1e-9 * e0, (g, n)


def test_driving_full_chain_p13_every_step(driving, driving_full_p75):
    """P13 certificates at every step of the rank-512 chain at 75% pruning,
    all four gates: (ii) the exported unpruned v_n and u_n are the top
    singular pair of the residual the earlier terms leave, ||R v_n - sigma_n
    u_n|| and ||R^T u_n - sigma_n v_n|| <= 1e-10 sigma_1; (iii) the stored
    mask equals the NZ largest magnitudes of v_n (lower index first on
    ties), bit-exactly (Sec. III: prune(v, NZ) of Eq. (1))."""
    m = driving_full_p75
    W = driving.W.astype(np.float64)
    for g in range(4):
        R = W[g * 512:(g + 1) * 512].copy()
        lf = B.approx_lstm_get_factors(m, g)
        l64 = B.approx_lstm_get_factors_f64(m, g)
        sig, U, V = l64["sigma"], l64["u"], l64["v"]
        idx = lf["v_idx"].astype(np.int64)
        s1 = sig[0]
        worst = 0.0
        for n in range(512):
            mask = oracle.magnitude_mask(V[n], 640)
            assert np.array_equal(mask, idx[n]), (g, n)
            r1 = np.linalg.norm(R @ V[n] - sig[n] * U[n])
            r2 = np.linalg.norm(R.T @ U[n] - sig[n] * V[n])
            worst = max(worst, r1, r2)
            assert r1 <= 1e-10 * s1 and r2 <= 1e-10 * s1, (g, n, r1, r2)
            R[:, idx[n]] -= sig[n] * np.outer(U[n], V[n][idx[n]])
        print(f"gate {g}: worst singular-pair residual {worst / s1:.2e} sigma_1 over 512 steps")


def test_launch_plans_of_the_tested_shapes():
    """approx_lstm_plan (no device work) on host-only models: the shapes the
    GPU tests use reach the launch paths they are meant to cover, in
    particular P_x streamed one timestep ahead (px_all 0) on each exchange
    path and on a single workgroup, and the plan of the timed workload."""
    tiny = synth.make(64, 32, 600, 1, index=44, xkind="normal")
    m = prep(tiny, 32, p=0.5, flags=B.FLAG_HOST_ONLY)
    B.approx_lstm_set_launch(m, 2, 0)
    p = B.approx_lstm_plan(m, 600, 1, online=1, num_cu=256)
    assert (p["blocks"], p["px_all"], p["bulk_h"]) == (2, 0, 0), p
    p = B.approx_lstm_plan(m, 200, 1, online=1, num_cu=256)
    assert (p["blocks"], p["px_all"]) == (2, 1), p
    B.approx_lstm_set_launch(m, 1, 0)
    for online in (0, 1):
        p = B.approx_lstm_plan(m, 300, 1, [32], online=online, num_cu=256)
        assert (p["blocks"], p["px_all"]) == (1, 0), p
        p = B.approx_lstm_plan(m, 8, 1, [32], online=online, num_cu=256)
        assert (p["blocks"], p["px_all"]) == (1, 1), p
    B.approx_lstm_set_launch(m, 0, 0)
    p = B.approx_lstm_plan(m, 8, 1, [0, 1, 4, 16, 32], num_cu=256)
    assert p["allpairs"] == 1 and p["px_all"] == 1, p
    wide = synth.make(512, 512, 48, 8, index=43, xkind="relu")
    m2 = prep(wide, 128, p=0.75, flags=B.FLAG_HOST_ONLY)
    B.approx_lstm_set_launch(m2, 8, 0)
    p = B.approx_lstm_plan(m2, 48, 8, online=1, num_cu=256)
    assert (p["px_all"], p["bulk_h"], p["allpairs"]) == (0, 1, 1), p
    B.approx_lstm_set_launch(m2, 0, 0)
    p = B.approx_lstm_plan(m2, 48, 8, online=1, num_cu=256)
    assert (p["px_all"], p["bulk_h"], p["allpairs"]) == (1, 1, 1), p
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_plan(m2, 48, 8, [129], num_cu=256)
    assert ei.value.status == B.ERR_INVALID_ARG


def test_driving_plan_of_the_timed_workload(driving, driving_full_p75):
    """The timed workload (driving shape, K = 512, one sequence, T = 16) on
    256 compute units: P_x of every timestep resident, register-resident
    h-part entries and U rows, tagged h words."""
    p = B.approx_lstm_plan(driving_full_p75, 16, 1, [512], num_cu=256)
    assert p["px_all"] == 1 and p["bulk_h"] == 0 and p["hpl"] > 0 and p["upt"] > 0, p
    assert p["lds_bytes"] <= 160 * 1024, p
    assert p["pair_kernel"] == 1 and p["blocks"] > 1, p


def test_driving_small_budgets_take_one_workgroup(driving_full_p75):
    """Budgets up to K = 16 at the driving shape fit one workgroup's
    registers (two phase-A passes, four output rows per thread): nothing is
    exchanged between workgroups.  K = 32 needs more than one."""
    for K in (1, 2, 4, 8, 16):
        p = B.approx_lstm_plan(driving_full_p75, 16, 1, [K], num_cu=256)
        assert p["pair_kernel"] == 1 and p["blocks"] == 1, (K, p)
    p = B.approx_lstm_plan(driving_full_p75, 16, 1, [32], num_cu=256)
    assert p["pair_kernel"] == 1 and p["blocks"] > 1, p


def test_driving_pair_widths(driving_full_p75):
    """One-pair launch widths at the driving shape on 256 compute units: at
    least 16 workgroups from 17 terms per group and 32 from 64 (below that
    the narrowest width leaves hundreds of rows per workgroup), 64 at the
    timed K = 512, one workgroup up to 16 terms."""
    want = {1: 1, 16: 1, 17: 16, 32: 16, 63: 16, 64: 32, 128: 32, 256: 32, 512: 64}
    for K, P in want.items():
        p = B.approx_lstm_plan(driving_full_p75, 16, 1, [K], num_cu=256)
        assert p["pair_kernel"] == 1 and p["blocks"] == P, (K, p)
    # a smaller device caps the floor
    p = B.approx_lstm_plan(driving_full_p75, 16, 1, [64], num_cu=8)
    assert p["blocks"] <= 8, p


def test_driving_no_pruning_gives_the_svd(driving):
    """NZ = C: the chain is the SVD of each gate (P4), over all 512 steps."""
    m = prep(driving, 512, p=0.0)
    W = driving.W.astype(np.float64)
    for g in range(4):
        S = np.linalg.svd(W[g * 512:(g + 1) * 512], compute_uv=False)
        l64 = B.approx_lstm_get_factors_f64(m, g)
        np.testing.assert_allclose(l64["sigma"], S, rtol=1e-10)
        lf = B.approx_lstm_get_factors(m, g)
        assert np.array_equal(lf["v_idx"], np.tile(np.arange(2560), (512, 1)))


def test_termination_and_zero_matrix():
    D, H = 6, 2
    W = np.zeros((8, 8), np.float32)
    m = B.approx_lstm_prepare(W[:, :D], W[:, D:], None, D, H, 3, nz=4, flags=HOST)
    assert m.info["eff_rank"] == [0, 0, 0, 0]
    lf = B.approx_lstm_get_factors(m, 0)
    assert np.all(lf["sigma"] == 0) and np.all(lf["v_idx"] == np.arange(4))


def test_nz_from_ratio_matches_oracle():
    for D, H, p in [(64, 32, .5), (2048, 512, .9), (40, 23, .33), (17, 3, .999)]:
        rng = np.random.default_rng(1)
        W = rng.normal(size=(4 * H, D + H)).astype(np.float32)
        m = B.approx_lstm_prepare(W[:, :D], W[:, D:], None, D, H, 1, prune_ratio=p, flags=HOST)
        assert m.info["nz"] == oracle.nz_from_ratio(D + H, p)


@pytest.mark.parametrize("kw,status", [
    (dict(rank=0), B.ERR_INVALID_ARG),
    (dict(groups=2), B.ERR_INVALID_ARG),
    (dict(nz=97), B.ERR_INVALID_ARG),
    (dict(nz=-1), B.ERR_INVALID_ARG),
    (dict(prune_ratio=1.0), B.ERR_INVALID_ARG),
    (dict(factor_dtype=2), B.ERR_INVALID_ARG),
])
def test_prepare_rejects_bad_arguments(kw, status):
    w = synth.named("tiny")
    args = dict(rank=4, nz=0, prune_ratio=0.5, groups=4, flags=HOST)
    args.update(kw)
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_prepare(w.W[:, :64], w.W[:, 64:], w.b, 64, 32, **args)
    assert ei.value.status == status
    assert B.approx_lstm_last_error()


@pytest.mark.parametrize("G", [4, 1])
def test_bf16_model_stores_rounded_values_of_the_same_chain(G):
    """factor_dtype 1: the masks are those of the fp32 model (decided in fp64
    before rounding), sigma stays fp32, and u and the v values are the fp64
    values rounded fp64 -> fp32 -> bf16 (nearest even), as the oracle rounds."""
    w = synth.named("tiny")
    m32 = prep(w, 96, p=0.5, groups=G)
    m16 = B.approx_lstm_prepare(w.W[:, :64], w.W[:, 64:], w.b, 64, 32, 96, prune_ratio=0.5, groups=G,
                                flags=HOST, factor_dtype=1)
    assert m16.info["factor_dtype"] == 1 and m32.info["factor_dtype"] == 0
    for g in range(G):
        a, b = B.approx_lstm_get_factors(m32, g), B.approx_lstm_get_factors(m16, g)
        l64 = B.approx_lstm_get_factors_f64(m16, g)
        assert np.array_equal(a["v_idx"], b["v_idx"])
        assert np.array_equal(a["sigma"], b["sigma"])
        assert np.array_equal(b["u"], oracle.round_bf16(l64["u"]).astype(np.float32))
        vsel = np.take_along_axis(l64["v"], b["v_idx"].astype(np.int64), axis=1)
        assert np.array_equal(b["v_val"], oracle.round_bf16(vsel).astype(np.float32))
        assert not np.array_equal(a["u"], b["u"])


def test_host_only_model_cannot_run():
    w = synth.named("tiny")
    m = prep(w, 4, p=0.5)
    assert m.info["has_device_store"] == 0
    lv = (B.ctypes.c_int32 * 1)(1)
    st = B.lib.approx_lstm_run(m.handle, None, 1, 1, None, None, lv, 1, None, None, None)
    assert st == B.ERR_INVALID_ARG


def test_too_wide_input_is_unsupported():
    D, H = 65530, 8
    with pytest.raises(B.ApproxLstmError) as ei:
        B.approx_lstm_prepare(np.zeros((32, D), np.float32), np.zeros((32, H), np.float32), None,
                              D, H, 1, nz=1, flags=HOST)
    assert ei.value.status == B.ERR_UNSUPPORTED


@pytest.mark.parametrize("G", [4, 1])
def test_non_residual_ablation_matches_oracle(G):
    """APPROX_LSTM_FLAG_NON_RESIDUAL (Sec. III's alternative): the library's
    terms equal the oracle's residual=False terms, masks bit-exact over the
    tiny workload's chain (up to the rank of the gate matrix, where the
    spectrum ends)."""
    w = synth.named("tiny")
    nz = oracle.nz_from_ratio(96, 0.5)
    rank = 32 if G == 4 else 96
    m = prep(w, rank, p=0.5, groups=G, flags=HOST | B.FLAG_NON_RESIDUAL)
    f = oracle.prepare(w.W, 32, rank, nz, groups=G, residual=False)
    assert m.info["eff_rank"] == list(f.eff_rank)
    for g in range(G):
        lf = B.approx_lstm_get_factors(m, g)
        l64 = B.approx_lstm_get_factors_f64(m, g)
        assert np.array_equal(lf["v_idx"], f.mask[g])
        np.testing.assert_allclose(l64["sigma"], f.sigma[g], rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(l64["v"], f.v_full[g], atol=1e-9)


def test_non_residual_driving_prefix():
    w = synth.named("driving")
    nz = oracle.nz_from_ratio(2560, 0.75)
    m = prep(w, 24, p=0.75, flags=HOST | B.FLAG_NON_RESIDUAL)
    f = oracle.prepare(w.W, 512, 24, nz, residual=False)
    for g in range(4):
        assert np.array_equal(B.approx_lstm_get_factors(m, g)["v_idx"], f.mask[g]), g


def test_device_factorise_and_host_only_exclude_each_other():
    """Flag check before any device work (runs without a GPU)."""
    w = synth.named("tiny")
    with pytest.raises(B.ApproxLstmError) as ei:
        prep(w, 4, p=0.5, flags=B.FLAG_HOST_ONLY | B.FLAG_DEVICE_FACTORISE)
    assert ei.value.status == B.ERR_INVALID_ARG


def test_host_only_model_rejects_every_run_mode():
    """A model without a device store: run, deadline and anytime modes all
    refuse it with INVALID_ARG, before touching a device."""
    w = synth.named("tiny")
    m = prep(w, 8, p=0.5)
    for fn in ("approx_lstm_run_deadline", "approx_lstm_run_anytime"):
        st = getattr(B.lib, fn)(m.handle, None, 2, 1, None, None, 10.0, None, None, None, None)
        assert st == B.ERR_INVALID_ARG, fn


def test_batched_path_selector_arguments():
    """approx_lstm_set_batched_path accepts 0..3 and refuses anything else or a
    null model (a setting only: no device work)."""
    w = synth.named("tiny")
    m = prep(w, 4, p=0.5)
    for mode in (0, 1, 2, 3, 1):
        assert B.lib.approx_lstm_set_batched_path(m.handle, mode) == B.OK
    for mode in (-1, 4):
        assert B.lib.approx_lstm_set_batched_path(m.handle, mode) == B.ERR_INVALID_ARG
    assert B.lib.approx_lstm_set_batched_path(None, 1) == B.ERR_INVALID_ARG
