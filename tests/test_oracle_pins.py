"""Pins of the float64 oracle against things other than itself: library
routines, closed forms, invariants, brute force and the paper's printed
numbers.  Each test names the property it checks and the passage that fixes
it; a plausible mistake in the oracle (a dropped term, a wrong sign or index,
a transposed operand) should fail at least one of them.  CPU only."""

import itertools
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle.factorise import fix_sign
from paper_1905_00689_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_lstm(D, H, seed, scale=None):
    rng = np.random.default_rng(seed)
    C = D + H
    s = 1.0 / math.sqrt(C) if scale is None else scale
    W = rng.normal(0, s, size=(4 * H, C))
    b = rng.normal(0, 0.1, size=4 * H)
    return W, b, rng


# --------------------------------------------------------------------- P1
@pytest.mark.parametrize("D,H,T,B", [(5, 3, 4, 2), (64, 32, 8, 1), (17, 9, 6, 3)])
def test_p1_exact_lstm_matches_torch_lstm(D, H, T, B):
    """Sec. II / Fig. 1 gate structure: the exact recurrence equals
    torch.nn.LSTM in float64 (gate rows i, f, g, o; bias_hh = 0)."""
    W, b, rng = rand_lstm(D, H, 11 + D)
    x = rng.normal(size=(T, B, D))
    h0 = rng.normal(size=(B, H))
    c0 = rng.normal(size=(B, H))
    lstm = torch.nn.LSTM(D, H).double()
    with torch.no_grad():
        lstm.weight_ih_l0.copy_(torch.from_numpy(W[:, :D]))
        lstm.weight_hh_l0.copy_(torch.from_numpy(W[:, D:]))
        lstm.bias_ih_l0.copy_(torch.from_numpy(b))
        lstm.bias_hh_l0.zero_()
        out, (hT, cT) = lstm(torch.from_numpy(x), (torch.from_numpy(h0)[None], torch.from_numpy(c0)[None]))
    hs, c = oracle.exact_lstm(W, b, x, h0, c0)
    np.testing.assert_allclose(hs, out.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(c, cT[0].numpy(), rtol=0, atol=1e-12)


def test_sigmoid_is_stable_and_matches_definition():
    z = np.array([-800.0, -30.0, -1.0, 0.0, 1.0, 30.0, 800.0])
    s = oracle.sigmoid(z)
    assert np.all(np.isfinite(s))
    np.testing.assert_allclose(s[1:-1], 1.0 / (1.0 + np.exp(-z[1:-1])), rtol=1e-15)
    assert s[0] == 0.0 and s[-1] == 1.0


# --------------------------------------------------------------- triplet
@pytest.mark.parametrize("shape", [(6, 10), (10, 6), (32, 96), (128, 96), (7, 7)])
def test_top_triplet_matches_lapack_svd(shape):
    """The top singular triplet equals numpy.linalg.svd's first triplet (up to sign)."""
    rng = np.random.default_rng(shape[0] * 100 + shape[1])
    R = rng.normal(size=shape)
    s, u, v = oracle.top_triplet(R)
    U, S, Vt = np.linalg.svd(R)
    assert abs(s - S[0]) <= 1e-12 * S[0]
    sign = np.sign(u @ U[:, 0])
    np.testing.assert_allclose(sign * u, U[:, 0], atol=1e-10)
    np.testing.assert_allclose(sign * v, Vt[0], atol=1e-10)
    # singular-triplet equations hold to rounding
    assert np.linalg.norm(R @ v - s * u) <= 1e-12 * S[0]
    assert np.linalg.norm(R.T @ u - s * v) <= 1e-12 * S[0]


def test_fix_sign_rule():
    u = np.array([1.0, 2.0])
    v = np.array([0.5, -3.0, 3.0, 1.0])          # tie on |v| at 1 and 2: lowest index wins
    u2, v2 = fix_sign(u, v)
    assert v2[1] == 3.0 and np.all(u2 == -u)
    u3, v3 = fix_sign(u, -v)
    assert v3[1] == 3.0 and np.all(u3 == u)


# --------------------------------------------------------------------- P3
@pytest.mark.parametrize("C,nz", [(8, 3), (10, 5), (12, 4), (9, 1), (7, 7)])
def test_p3_mask_is_optimal_by_brute_force(C, nz):
    """Sec. III magnitude pruning: over every mask of size NZ, the kept
    largest-magnitude entries maximise ||v * m||^2 and hence minimise the
    one-step residual ||R - sigma u (v*m)^T||_F."""
    rng = np.random.default_rng(C * 7 + nz)
    R = rng.normal(size=(5, C))
    s, u, v = oracle.top_triplet(R)
    m = oracle.magnitude_mask(v, nz)
    assert list(m) == sorted(m) and len(set(m)) == nz
    best = None
    for sub in itertools.combinations(range(C), nz):
        vm = np.zeros(C)
        vm[list(sub)] = v[list(sub)]
        r = np.linalg.norm(R - s * np.outer(u, vm))
        if best is None or r < best[0] - 1e-12:
            best = (r, sub)
    vm = np.zeros(C)
    vm[m] = v[m]
    assert np.linalg.norm(R - s * np.outer(u, vm)) <= best[0] + 1e-12
    assert tuple(m) == best[1]


def test_mask_ties_go_to_lower_index():
    v = np.array([1.0, -2.0, 2.0, 0.5, -2.0, 1.0])
    assert list(oracle.magnitude_mask(v, 2)) == [1, 2]
    assert list(oracle.magnitude_mask(v, 4)) == [0, 1, 2, 4]
    assert list(oracle.magnitude_mask(v, 6)) == [0, 1, 2, 3, 4, 5]


# --------------------------------------------------------------------- P2
@pytest.mark.parametrize("G,nz", [(4, 48), (1, 48), (4, 10), (1, 96)])
def test_p2_residual_energy_identity(G, nz):
    """Residual definition after Eq. (1): R^(n+1) = R^(n) - sigma u prune(v)^T.
    Since u^T R = sigma v^T, ||R^(n+1)||_F^2 = ||R^(n)||_F^2 - sigma^2 ||v'||^2,
    so the approximation error is non-increasing in the number of steps.  The
    trajectory is also recomputed from the stored terms (W - W~^(n))."""
    w = synth.named("tiny")
    W = w.W.astype(np.float64)
    f = oracle.prepare(W, 32, 40, nz, groups=G, record_trajectory=True)
    Rg = f.rows
    for g in range(G):
        tr = f.trajectory[g]
        Wg = W[g * Rg:(g + 1) * Rg]
        for n in range(len(tr) - 1):
            vp2 = np.sum(f.vals[g, n] ** 2)
            pred = tr[n] - f.sigma[g, n] ** 2 * vp2
            assert abs(tr[n + 1] - pred) <= 1e-10 * tr[0]
            assert tr[n + 1] <= tr[n] * (1 + 1e-12)
        for K in (0, 1, 5, 17, len(tr) - 1):
            err = np.sum((Wg - oracle.reconstruct(f, g, K)) ** 2)
            assert abs(err - tr[K]) <= 1e-10 * tr[0]


# --------------------------------------------------------------------- P4
@pytest.mark.parametrize("G", [4, 1])
def test_p4_no_pruning_is_truncated_svd_and_exact_at_full_rank(G):
    """With NZ = C the residual scheme is the SVD: sigma_n are W_g's singular
    values, W~^(K) is the best rank-K approximation (Eckart-Young) and at
    K >= rank the progressive LSTM equals the exact one."""
    w = synth.named("tiny")
    W = w.W.astype(np.float64)
    H, C = 32, 96
    f = oracle.prepare(W, H, 96, C, groups=G)
    Rg = f.rows
    for g in range(G):
        Wg = W[g * Rg:(g + 1) * Rg]
        S = np.linalg.svd(Wg, compute_uv=False)
        r = min(Wg.shape)
        assert f.eff_rank[g] == r
        np.testing.assert_allclose(f.sigma[g, :r], S, rtol=1e-10)
        assert np.all(f.sigma[g, r:] == 0) and np.all(f.U[g, r:] == 0)
        for K in (1, 3, 10, r):
            err = np.sum((Wg - oracle.reconstruct(f, g, K)) ** 2)
            assert abs(err - np.sum(S[K:] ** 2)) <= 1e-10 * np.sum(S ** 2)
    hs, cs = oracle.run(f, w.b, w.x, [96])
    he, ce = oracle.exact_lstm(W, w.b, w.x)
    np.testing.assert_allclose(hs[0], he, atol=1e-12)
    np.testing.assert_allclose(cs[0], ce, atol=1e-12)


# --------------------------------------------------------------------- P5
@pytest.mark.parametrize("nz", [1, 3, 7])
def test_p5_single_row_reduces_to_magnitude_sorting(nz):
    """R_g = 1 (H = 1, per-gate groups): each residual is one row, its top
    triplet is the row itself, so after n steps W~ is w restricted to its
    n*NZ largest-magnitude entries (ties to the lower index)."""
    D, H = 20, 1
    W, b, rng = rand_lstm(D, H, 5)
    C = D + H
    f = oracle.prepare(W, H, 10, nz, groups=4)
    for g in range(4):
        w = W[g]
        order = np.lexsort((np.arange(C), -np.abs(w)))
        for n in range(1, 4):
            keep = order[:min(n * nz, C)]
            expect = np.zeros(C)
            expect[keep] = w[keep]
            np.testing.assert_allclose(oracle.reconstruct(f, g, n)[0], expect, atol=1e-13)


# --------------------------------------------------------------------- P6
def test_p6_zero_budget_closed_form():
    """K = 0 leaves only the bias: with h0 = c0 = 0 the gates are constant, so
    c_t = i * g * (1 - f^t) / (1 - f) and h_t = o * tanh(c_t)."""
    w = synth.named("tiny")
    f = oracle.prepare(w.W, 32, 4, 48, groups=4)
    hs, _ = oracle.run(f, w.b, w.x, [0])
    b = w.b.astype(np.float64)
    H = 32
    sg = lambda z: 1 / (1 + np.exp(-z))
    i, fg, g, o = sg(b[:H]), sg(b[H:2 * H]), np.tanh(b[2 * H:3 * H]), sg(b[3 * H:])
    for t in range(w.T):
        c = i * g * (1 - fg ** (t + 1)) / (1 - fg)
        np.testing.assert_allclose(hs[0, t, 0], o * np.tanh(c), atol=1e-14)


# --------------------------------------------------------------------- P7
def test_p7_rank_one_gate_is_exact_after_one_step():
    """A gate matrix a b^T with nnz(b) <= NZ is recovered by one refinement step."""
    D, H = 12, 4
    rng = np.random.default_rng(3)
    C = D + H
    W = np.zeros((4 * H, C))
    for g in range(4):
        a = rng.normal(size=H)
        bb = np.zeros(C)
        idx = rng.choice(C, 5, replace=False)
        bb[idx] = rng.normal(size=5)
        W[g * H:(g + 1) * H] = np.outer(a, bb)
    f = oracle.prepare(W, H, 3, 5, groups=4)
    assert list(f.eff_rank) == [1, 1, 1, 1]
    x = rng.normal(size=(5, 2, D))
    bias = rng.normal(size=4 * H)
    hs, _ = oracle.run(f, bias, x, [1])
    he, _ = oracle.exact_lstm(W, bias, x)
    np.testing.assert_allclose(hs[0], he, atol=1e-13)


# --------------------------------------------------------------------- P8
@pytest.mark.parametrize("nz", [5, 24, 96])
def test_p8_geometric_decay_bound(nz):
    """||v'||^2 >= NZ/C (top-NZ of a unit vector) and sigma^2 >= ||R||_F^2 / rank,
    so each step removes at least a fraction NZ/(C*min(R_g,C)) of the residual energy."""
    w = synth.named("tiny")
    f = oracle.prepare(w.W, 32, 30, nz, groups=4, record_trajectory=True)
    C, Rg = 96, 32
    q = 1 - nz / (C * min(Rg, C))
    for g in range(4):
        tr = f.trajectory[g]
        for n in range(len(tr) - 1):
            assert np.sum(f.vals[g, n] ** 2) >= nz / C - 1e-12
            assert tr[n + 1] <= q * tr[n] + 1e-12 * tr[0]


# --------------------------------------------------------------------- P9
def test_p9_equivariances():
    """Permuting input features permutes mask indices and leaves h unchanged;
    permuting hidden units permutes h; scaling W by a > 0 scales sigma and keeps
    the masks."""
    D, H, T, B = 10, 4, 5, 2
    W, b, rng = rand_lstm(D, H, 21)
    x = rng.normal(size=(T, B, D))
    nz, N = 6, 8
    f = oracle.prepare(W, H, N, nz)
    h, _ = oracle.run(f, b, x, [3, 8])
    # input permutation
    p = rng.permutation(D)
    Wp = np.concatenate([W[:, :D][:, p], W[:, D:]], axis=1)
    fp = oracle.prepare(Wp, H, N, nz)
    hp, _ = oracle.run(fp, b, x[:, :, p], [3, 8])
    np.testing.assert_allclose(hp, h, atol=1e-11)
    colmap = np.concatenate([np.argsort(p), np.arange(D, D + H)])   # new index of old column
    for g in range(4):
        for n in range(N):
            assert sorted(colmap[f.mask[g, n]]) == list(fp.mask[g, n])
    # hidden-unit permutation (rows within each gate and the W_hh columns)
    q = rng.permutation(H)
    rows = np.concatenate([g * H + q for g in range(4)])
    Wq = W[rows][:, np.concatenate([np.arange(D), D + q])]
    fq = oracle.prepare(Wq, H, N, nz)
    hq, _ = oracle.run(fq, b[rows], x, [3, 8])
    np.testing.assert_allclose(hq, h[..., q], atol=1e-11)
    # positive scaling
    fs = oracle.prepare(2.5 * W, H, N, nz)
    np.testing.assert_allclose(fs.sigma, 2.5 * f.sigma, rtol=1e-11)
    assert np.array_equal(fs.mask, f.mask)


# -------------------------------------------------------------------- P10
def test_p10_levels_are_independent_recurrences():
    w = synth.named("tiny")
    f = oracle.prepare(w.W, 32, 20, 48)
    hs, cs = oracle.run(f, w.b, w.x, [0, 4, 20])
    for j, K in enumerate([0, 4, 20]):
        h1, c1 = oracle.run(f, w.b, w.x, [K])
        assert np.array_equal(h1[0], hs[j]) and np.array_equal(c1[0], cs[j])
    hsched, _ = oracle.run_schedule(f, w.b, w.x, [4] * w.T)
    assert np.array_equal(hsched, hs[1])


# -------------------------------------------------------------------- P11
@pytest.mark.parametrize("G,nz", [(4, 48), (1, 48), (4, 96)])
def test_p11_output_error_trends_down_with_budget(G, nz):
    """Refinement steps improve the output on the tiny workload: the error is
    ~0 at full rank without pruning and the Kendall tau between K and the h
    error is clearly negative (the paper notes the trade-off need not be
    monotone, so only the trend is checked)."""
    from scipy.stats import kendalltau
    w = synth.named("tiny")
    f = oracle.prepare(w.W, 32, 96, nz, groups=G)
    Ks = [0, 1, 2, 4, 8, 16, 24, 32, 48, 64, 96]
    hs, _ = oracle.run(f, w.b, w.x, Ks)
    he, _ = oracle.exact_lstm(w.W, w.b, w.x)
    errs = [np.abs(hs[j] - he).max() for j in range(len(Ks))]
    tau, _ = kendalltau(Ks, errs)
    assert tau < -0.5
    if nz == 96:
        assert errs[-1] < 1e-12


# -------------------------------------------------------------------- P12
def _table1():
    rows = {}
    with open(os.path.join(GOLDEN, "table1_platforms.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            plat, bench, lat, pw, eff = line.split()
            rows[bench if bench != "baseline" else plat] = (float(lat), float(pw), float(eff))
    return rows


def test_p12_opcounts_and_table1_arithmetic():
    """Sec. III: N_steps*(2R+2NZ+1) ops per gate; Sec. VI-B.1: 2RC for the dense
    gate.  Table I's efficiency column is 4*2RC dense-equivalent ops per
    timestep / latency / power (R=64, C=8320) to within the printed digits."""
    assert oracle.gate_ops_dense(64, 8320) == 1064960
    assert oracle.gate_ops_progressive(64, 4160, 1) == 2 * 64 + 2 * 4160 + 1
    assert oracle.gate_ops_progressive(64, 130, 10) == 10 * (128 + 260 + 1)
    for name, (lat, pw, eff) in _table1().items():
        got = oracle.table1_efficiency(lat, pw)
        assert abs(got - eff) / eff < 2e-3, (name, got, eff)


def test_p12_stated_speedups_follow_table1():
    t = _table1()
    with open(os.path.join(GOLDEN, "speedups_sec6b.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            prop, base, ratio = line.split()
            got = t[base][0] / t[prop][0]
            assert abs(got - float(ratio)) / float(ratio) < 0.02, (prop, base, got)


# ------------------------------------------------------------- NZ, bf16
def test_nz_from_ratio_matches_workload_table():
    for C, p, nz in [(96, .5, 48), (2560, 0, 2560), (2560, .5, 1280), (2560, .75, 640),
                     (2560, .9, 256), (5120, .75, 1280), (2048, .75, 512), (4096, .9, 410)]:
        assert oracle.nz_from_ratio(C, p) == nz


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(9)
    a = np.concatenate([rng.normal(size=5000) * 10.0 ** rng.integers(-20, 20, 5000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, -3.3e-39]])
    ref = torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(oracle.round_bf16(a), ref)


def test_bf16_operands_are_a_no_op_when_every_operand_is_representable():
    """Batched bf16 configuration: rounding x~ and z to bf16 changes nothing
    when they are already bf16 values.  Each gate is 4 u e_k^T with u having
    entries +-1/2 (so sigma = 4, v = e_k, one kept entry) and x on a grid of
    1/8: after one step the bf16-operand run, the plain run and the exact
    LSTM coincide."""
    D, H = 6, 4
    W = np.zeros((4 * H, D + H))
    signs = np.array([[1, -1, 1, 1], [-1, -1, 1, -1], [1, 1, -1, 1], [-1, 1, 1, 1]]) * 0.5
    for g, k in enumerate([0, 2, 3, 5]):
        W[g * H:(g + 1) * H, k] = 4.0 * signs[g]
    b = np.array([0.125, -0.25, 0.5, 0.0] * 4)
    x = np.array([[[0.125, -1.5, 2.0, 0.375, 0.0, -0.625]]])
    f = oracle.prepare(W, H, 1, 1).rounded("bf16")
    assert np.allclose(f.sigma, 4.0) and np.all(f.mask[:, 0, 0] == [0, 2, 3, 5])
    h16, c16 = oracle.run(f, b, x, [1], operand_round="bf16")
    h64, c64 = oracle.run(f, b, x, [1])
    he, ce = oracle.exact_lstm(W, b, x)
    assert np.array_equal(h16, h64) and np.array_equal(c16, c64)
    np.testing.assert_allclose(h64[0], he, rtol=0, atol=1e-15)


def test_bf16_operand_error_within_the_rounding_bound():
    """Batched bf16 configuration, one timestep from h0 = c0 = 0: each
    product takes three rounded quantities (v value, x~ entry, then z with u),
    so |dy| <= ((1 + 2^-8)^3 - 1) * sum_n |sigma_n| |u_n| (|v'_n|^T |x~|) to first
    order, with 2^-8 bounding bf16's relative rounding error; the cell update
    then gives |dh| <= (1/4 + 1/4 + 1) max |dy| (sigmoid' <= 1/4, tanh' <= 1).
    The bf16 mode must differ from the fp64 mode, and by no more than that."""
    w = synth.named("tiny")
    f = oracle.prepare(w.W, 32, 96, 48).rounded("bf16")
    x1 = w.x[:1].astype(np.float64)
    h16, _ = oracle.run(f, w.b, x1, [96], operand_round="bf16")
    h64, _ = oracle.run(f, w.b, x1, [96])
    xt = np.abs(np.concatenate([x1[0], np.zeros((1, 32))], axis=1))[0]
    bound = np.zeros(128)
    for g in range(4):
        V = np.abs(oracle.dense_pruned_v(f, g))
        bound[g * 32:(g + 1) * 32] = (np.abs(f.U[g]).T * np.abs(f.sigma[g])) @ (V @ xt)
    u = 2.0 ** -8
    dy = ((1 + u) ** 3 - 1) * bound
    diff = np.abs(h16 - h64).max()
    assert 0 < diff <= 1.5 * dy.max()


def test_bf16_rounds_z_itself_hand_worked():
    """Where the bf16 configuration rounds (Q14 reading of Eq. (1) with bf16
    operands): z = sigma * s, then z is rounded before it meets u.  One
    timestep, H = 1, each gate's 1 x 3 block sigma_g u_g e_0^T (so v = e_0,
    one kept entry, u = +-1, sigma in {3, 5, 7}: all bf16 values), x_0 =
    1 + 2^-7 (a bf16 value), h0 = c0 = 0, so s = x_0 and sigma * s is exact in
    float64 but needs 9 significant bits.  Worked by hand, nearest even at 8
    bits:
        3 * (1 + 2^-7) = 11.0000011b -> tie, odd kept bit  -> 11.000010b = 3.03125
        5 * (1 + 2^-7) = 101.0000101b -> below half        -> 101.00001b = 5.03125
        7 * (1 + 2^-7) = 111.0000111b -> above half        -> 111.00010b = 7.0625
    so the gate pre-activations are b_g + u_g * z16_g exactly, and the run
    must equal the exact LSTM with zero weights and that bias.  Not rounding
    z, or rounding y = b + z u instead of z, gives different outputs (the
    biases are chosen so that those roundings disagree)."""
    x0 = 1.0 + 2.0 ** -7
    sig = np.array([3.0, 5.0, 3.0, 7.0])
    u = np.array([1.0, -1.0, 1.0, 1.0])
    z16 = np.array([3.03125, 5.03125, 3.03125, 7.0625])
    b = np.array([2.0 ** -8, -0.75, 0.5, 2.0 ** -7])
    W = np.zeros((4, 3))
    W[:, 0] = sig * u
    x = np.array([[[x0, 0.5]]])
    assert np.array_equal(oracle.round_bf16(sig * x0), z16)
    f = oracle.prepare(W, 1, 1, 1).rounded("bf16")
    assert np.array_equal(f.sigma[:, 0], sig) and np.all(f.mask[:, 0, 0] == 0)
    assert np.array_equal(f.U[:, 0, 0], u) and np.array_equal(f.vals[:, 0, 0], np.ones(4))
    h16, c16 = oracle.run(f, b, x, [1], operand_round="bf16")
    zeros = np.zeros((4, 3))
    he, ce = oracle.exact_lstm(zeros, b + u * z16, x)
    assert np.array_equal(h16[0], he) and np.array_equal(c16[0], ce)
    h_unrounded, _ = oracle.exact_lstm(zeros, b + u * sig * x0, x)
    h_late, _ = oracle.exact_lstm(zeros, oracle.round_bf16(b + u * sig * x0), x)
    assert not np.array_equal(h16[0], h_unrounded)
    assert not np.array_equal(h16[0], h_late)


def test_termination_and_degenerate_zero_matrix():
    """A zero gate matrix has no live terms (every sigma 0, output bias-only)."""
    D, H = 6, 2
    W = np.zeros((4 * H, D + H))
    f = oracle.prepare(W, H, 3, 4)
    assert list(f.eff_rank) == [0, 0, 0, 0]
    assert np.all(f.sigma == 0) and np.all(f.U == 0)
    assert all(list(f.mask[g, n]) == [0, 1, 2, 3] for g in range(4) for n in range(3))


@pytest.mark.parametrize("G,nz,K", [(4, 48, 5), (1, 48, 7), (4, 10, 30), (1, 30, 96)])
def test_progressive_run_equals_exact_lstm_of_the_approximate_matrix(G, nz, K):
    """Eq. (1) evaluates W~^(K) x~ term by term, so the progressive recurrence
    equals the exact recurrence run with W~^(K) in place of W (ties run() to
    the approximation pinned by P2/P4/P5), including given h0 and c0."""
    w = synth.named("tiny")
    f = oracle.prepare(w.W, 32, 96, nz, groups=G)
    Rg = f.rows
    Wt = np.concatenate([oracle.reconstruct(f, g, K) for g in range(G)], axis=0)
    rng = np.random.default_rng(4)
    h0 = rng.normal(size=(1, 32))
    c0 = rng.normal(size=(1, 32))
    hs, cs = oracle.run(f, w.b, w.x, [K], h0, c0)
    he, ce = oracle.exact_lstm(Wt, w.b, w.x, h0, c0)
    np.testing.assert_allclose(hs[0], he, atol=1e-13)
    np.testing.assert_allclose(cs[0], ce, atol=1e-13)


# ------------------------------------------------------ row-tile baseline
def _torch_lstm(W, b, x, h0, c0):
    T, B, D = x.shape
    H = W.shape[0] // 4
    lstm = torch.nn.LSTM(D, H).double()
    with torch.no_grad():
        lstm.weight_ih_l0.copy_(torch.from_numpy(W[:, :D]))
        lstm.weight_hh_l0.copy_(torch.from_numpy(W[:, D:]))
        lstm.bias_ih_l0.copy_(torch.from_numpy(b))
        lstm.bias_hh_l0.zero_()
        out, (_, cT) = lstm(torch.from_numpy(x), (torch.from_numpy(h0)[None], torch.from_numpy(c0)[None]))
    return out.numpy(), cT[0].numpy()


@pytest.mark.parametrize("rows", [0, 1, 4, 8])
def test_row_tile_baseline_is_torch_lstm_with_unreached_rows_zeroed(rows):
    """Sec. VI-B row-tile baseline: after `rows` rows per gate, the output is
    the LSTM whose weight rows beyond that point (in every gate block i, f,
    g, o) are zero and whose bias is whole.  torch.nn.LSTM on the zeroed
    weights is an independent route to the same numbers; a wrong gate block
    or a bias dropped from an unreached row fails it."""
    D, H, T, B = 6, 8, 5, 3
    W, b, rng = rand_lstm(D, H, 401 + rows)
    x = rng.normal(size=(T, B, D))
    h0 = rng.normal(size=(B, H))
    c0 = rng.normal(size=(B, H))
    Wz = W.copy()
    for q in range(4):
        Wz[q * H + rows:(q + 1) * H] = 0.0
    he, ce = _torch_lstm(Wz, b, x, h0, c0)
    hs, c = oracle.row_tile_lstm(W, b, x, rows, h0, c0)
    np.testing.assert_allclose(hs, he, rtol=0, atol=1e-12)
    np.testing.assert_allclose(c, ce, rtol=0, atol=1e-12)


def test_row_tile_baseline_limits():
    """All rows reached is the exact LSTM; no row reached leaves the bias
    alone, whose recurrence from h0 = c0 = 0 has the closed form
    c_t = i g (1 - f^t) / (1 - f), h_t = o tanh(c_t)."""
    D, H, T, B = 7, 5, 6, 2
    W, b, rng = rand_lstm(D, H, 77)
    x = rng.normal(size=(T, B, D))
    hs, c = oracle.row_tile_lstm(W, b, x, H)
    he, ce = _torch_lstm(W, b, x, np.zeros((B, H)), np.zeros((B, H)))
    np.testing.assert_allclose(hs, he, rtol=0, atol=1e-12)
    np.testing.assert_allclose(c, ce, rtol=0, atol=1e-12)
    hs0, _ = oracle.row_tile_lstm(W, b, x, 0)
    sg = lambda z: 1 / (1 + np.exp(-z))
    i, fg, g, o = sg(b[:H]), sg(b[H:2 * H]), np.tanh(b[2 * H:3 * H]), sg(b[3 * H:])
    for t in range(T):
        ct = i * g * (1 - fg ** (t + 1)) / (1 - fg)
        for bb in range(B):
            np.testing.assert_allclose(hs0[t, bb], o * np.tanh(ct), atol=1e-14)


# ------------------------------------------------ non-residual alternative
@pytest.mark.parametrize("G", [4, 1])
def test_non_residual_terms_are_the_pruned_svd(G):
    """Sec. III's alternative to the residual scheme: the terms are the
    singular triplets of the original gate matrix (LAPACK SVD, sign rule
    applied), each v pruned on its own."""
    D, H = 10, 4
    W, _, _ = rand_lstm(D, H, 501)
    C, Rg = D + H, 4 * H // G
    nz = 5
    f = oracle.prepare(W, H, min(Rg, C), nz, groups=G, residual=False)
    for g in range(G):
        Ug, S, Vt = np.linalg.svd(W[g * Rg:(g + 1) * Rg])
        np.testing.assert_allclose(f.sigma[g], S[:min(Rg, C)], rtol=1e-12)
        for n in range(min(Rg, C)):
            u, v = fix_sign(Ug[:, n], Vt[n])
            np.testing.assert_allclose(f.U[g, n], u, atol=1e-10)
            np.testing.assert_allclose(f.v_full[g, n], v, atol=1e-10)
            assert np.array_equal(f.mask[g, n], oracle.magnitude_mask(v, nz))


def test_residual_and_non_residual_coincide_without_pruning():
    W, _, _ = rand_lstm(9, 3, 502)
    a = oracle.prepare(W, 3, 12, 12, residual=True)
    b = oracle.prepare(W, 3, 12, 12, residual=False)
    np.testing.assert_allclose(a.sigma, b.sigma, rtol=1e-10, atol=1e-14)
    assert np.array_equal(a.mask, b.mask)


def test_residual_scheme_has_lower_weight_error_than_non_residual():
    """The point of the residual scheme (Sec. III): with pruning, correcting
    the pruning error in later terms gives a smaller weight error at the same
    budget."""
    w = synth.named("tiny")
    a = oracle.prepare(w.W, 32, 32, 24, residual=True)
    b = oracle.prepare(w.W, 32, 32, 24, residual=False)
    W = w.W.astype(np.float64)
    for K in (8, 16, 32):
        ea = sum(np.linalg.norm(W[g * 32:(g + 1) * 32] - oracle.reconstruct(a, g, K)) ** 2 for g in range(4))
        eb = sum(np.linalg.norm(W[g * 32:(g + 1) * 32] - oracle.reconstruct(b, g, K)) ** 2 for g in range(4))
        assert ea < eb, (K, ea, eb)
