"""Parity of the exact (dense) LSTM path with the float64 oracle's exact LSTM.

The dense baseline computes the gate pre-activations with the full weight
matrices (Sec. II; no factorisation), so its reference is oracle.exact_lstm,
itself pinned to torch.nn.LSTM; the row-tile anytime baseline (Sec. VI-B, the
dense products stopped after a number of rows per gate) is compared with
oracle.row_tile_lstm.  Error measure and bar as for the fp32 progressive path
(1e-4).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1905_00689_amd import synth
from paper_1905_00689_amd import binding as B

from .gpu_helpers import rel_err, say

pytestmark = pytest.mark.gpu
TOL = 1e-4


def exact_model(w):
    return B.approx_lstm_exact_prepare(w.W[:, :w.D], w.W[:, w.D:], w.b, w.D, w.H)


def run_exact(m, x, h0=None, c0=None, want_c=False, rows=None):
    T, Bn, _ = x.shape
    H = m.hidden_size
    dev = torch.device("cuda")
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev)
    h = torch.full((T, Bn, H), float("nan"), device=dev)
    c = torch.full((Bn, H), float("nan"), device=dev) if want_c else None
    h0t = None if h0 is None else torch.from_numpy(np.ascontiguousarray(h0, np.float32)).to(dev)
    c0t = None if c0 is None else torch.from_numpy(np.ascontiguousarray(c0, np.float32)).to(dev)
    if rows is None:
        B.approx_lstm_exact_run(m, xt, h, h0t, c0t, c)
    else:
        B.approx_lstm_exact_run_rows(m, xt, rows, h, h0t, c0t, c)
    B.approx_lstm_exact_check(m)
    torch.cuda.synchronize()
    return h.cpu().numpy(), (c.cpu().numpy() if want_c else None)


@pytest.mark.parametrize("name", ["tiny", "driving"])
def test_exact_matches_oracle(name):
    w = synth.named(name)
    say("exact LSTM", name)
    h, _ = run_exact(exact_model(w), w.x)
    he, _ = oracle.exact_lstm(w.W, w.b, w.x)
    e = rel_err(h, he)
    say("  rel err", e)
    assert e < TOL


def test_exact_ragged_batch_state_and_launch_widths():
    """D=50, H=37 (hidden units split unevenly), 3 sequences with initial
    state; every launch width gives the same bits and the oracle's values."""
    w = synth.make(50, 37, 5, 3, index=31, xkind="relu")
    rng = np.random.default_rng(8)
    h0 = rng.normal(size=(3, 37)).astype(np.float32)
    c0 = rng.normal(size=(3, 37)).astype(np.float32)
    m = exact_model(w)
    he, ce = oracle.exact_lstm(w.W, w.b, w.x, h0, c0)
    ref = None
    for P in (0, 1, 3, 7, 37):
        say("exact ragged, blocks", P)
        B.approx_lstm_exact_set_launch(m, P)
        h, c = run_exact(m, w.x, h0, c0, want_c=True)
        assert rel_err(h, he) < TOL, P
        assert np.abs(c - ce).max() < TOL * max(1.0, np.abs(ce).max()), P
        if ref is None:
            ref = h
        else:
            assert np.array_equal(h, ref), P


def test_exact_deadline_workload_shape():
    """The deadline workload's shapes: D=2048, H=2048, T=64, 8 sequences."""
    w = synth.named("deadline")
    say("exact LSTM, deadline workload shape")
    h, _ = run_exact(exact_model(w), w.x)
    he, _ = oracle.exact_lstm(w.W, w.b, w.x)
    e = rel_err(h, he)
    say("  rel err", e)
    assert e < TOL


def test_exact_zero_length_and_errors():
    w = synth.named("tiny")
    m = exact_model(w)
    say("exact T=0 and argument errors")
    assert B.approx_lstm_exact_run(m, torch.zeros((0, 1, 64), device="cuda"),
                                   torch.zeros((0, 1, 32), device="cuda")) == B.OK
    with pytest.raises(TypeError):
        B.approx_lstm_exact_run(m, torch.zeros((2, 1, 64)), torch.zeros((2, 1, 32)))
    st = B.lib.approx_lstm_exact_run(m.handle, None, 2, 1, None, None, None, None, None)
    assert st == B.ERR_INVALID_ARG


@pytest.mark.parametrize("rows", [0, 1, 100, 256, 511])
def test_row_tile_baseline_matches_oracle(rows):
    """Driving workload shape (D=2048, H=512, T=16), the dense products
    stopped after `rows` rows of every gate."""
    w = synth.named("driving")
    say("row-tile baseline, driving shape, rows", rows)
    h, _ = run_exact(exact_model(w), w.x, rows=rows)
    he, _ = oracle.row_tile_lstm(w.W, w.b, w.x, rows)
    e = rel_err(h, he)
    say("  rel err", e)
    assert e < TOL


def test_row_tile_all_rows_is_the_exact_run_bit_for_bit():
    w = synth.named("driving")
    m = exact_model(w)
    say("row-tile rows = H against the exact run")
    h_rows, _ = run_exact(m, w.x, rows=w.H)
    h_full, _ = run_exact(m, w.x)
    assert np.array_equal(h_rows, h_full)


def test_row_tile_ragged_state_and_launch_widths():
    """D=50, H=37, 3 sequences with initial state: row budgets that end inside
    a workgroup's slice of units, every launch width giving the same bits."""
    w = synth.make(50, 37, 5, 3, index=32, xkind="relu")
    rng = np.random.default_rng(9)
    h0 = rng.normal(size=(3, 37)).astype(np.float32)
    c0 = rng.normal(size=(3, 37)).astype(np.float32)
    m = exact_model(w)
    for rows in (0, 5, 36):
        he, ce = oracle.row_tile_lstm(w.W, w.b, w.x, rows, h0, c0)
        ref = None
        for P in (1, 3, 7, 37):
            say("row-tile ragged, rows", rows, "blocks", P)
            B.approx_lstm_exact_set_launch(m, P)
            h, c = run_exact(m, w.x, h0, c0, want_c=True, rows=rows)
            assert rel_err(h, he) < TOL, (rows, P)
            assert np.abs(c - ce).max() < TOL * max(1.0, np.abs(ce).max()), (rows, P)
            if ref is None:
                ref = h
            else:
                assert np.array_equal(h, ref), (rows, P)


def test_row_tile_rejects_out_of_range_budgets():
    w = synth.named("tiny")
    m = exact_model(w)
    say("row-tile argument errors")
    x = torch.zeros((2, 1, 64), device="cuda")
    h = torch.zeros((2, 1, 32), device="cuda")
    for rows in (-1, 33):
        with pytest.raises(B.ApproxLstmError):
            B.approx_lstm_exact_run_rows(m, x, rows, h)


def test_exact_grouped_rows_ragged_batch():
    """H=600 (rows read from memory, not registers) with 11 sequences: each
    W_h row is applied to groups of 8 and 3 sequences.  Every launch width
    gives the same bits and the oracle's values; the row-tile variant too."""
    w = synth.make(40, 600, 4, 11, index=33, xkind="relu")
    rng = np.random.default_rng(10)
    h0 = rng.normal(size=(11, 600)).astype(np.float32)
    c0 = rng.normal(size=(11, 600)).astype(np.float32)
    m = exact_model(w)
    for rows in (None, 250):
        if rows is None:
            he, ce = oracle.exact_lstm(w.W, w.b, w.x, h0, c0)
        else:
            he, ce = oracle.row_tile_lstm(w.W, w.b, w.x, rows, h0, c0)
        ref = None
        for P in (0, 7, 75):
            say("exact grouped rows, rows", rows, "blocks", P)
            B.approx_lstm_exact_set_launch(m, P)
            h, c = run_exact(m, w.x, h0, c0, want_c=True, rows=rows)
            assert rel_err(h, he) < TOL, (rows, P)
            assert np.abs(c - ce).max() < TOL * max(1.0, np.abs(ce).max()), (rows, P)
            if ref is None:
                ref = h
            else:
                assert np.array_equal(h, ref), (rows, P)
