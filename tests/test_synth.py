"""The seeded input generators: shapes, determinism and the stated
distributions of the weight models (CPU only)."""

import numpy as np

from paper_1905_00689_amd import synth


def test_named_workloads_are_deterministic_and_shaped():
    for name in ("tiny", "driving", "paper"):
        a, b = synth.named(name), synth.named(name)
        assert np.array_equal(a.W, b.W) and np.array_equal(a.x, b.x)
        assert a.W.shape == (4 * a.H, a.D + a.H) and a.x.shape == (a.T, a.B, a.D)
        assert a.W.dtype == np.float32 and a.x.dtype == np.float32


def test_decay_model_has_unit_scale_blocks_with_decaying_spectra():
    w = synth.make(300, 20, 2, 1, index=99, wkind="decay")
    H = 20
    for q in range(4):
        blk = w.W[q * H:(q + 1) * H].astype(np.float64)
        assert abs(np.sum(blk * blk) - H) < 1e-3 * H
        s = np.linalg.svd(blk, compute_uv=False)
        assert np.all(np.diff(s) <= 1e-9) and s[0] > 4 * s[-1]
    # a few columns carry most of the weight: the heaviest 5% of columns hold
    # more than half of the squared norm
    cn = np.sort(np.sum(w.W.astype(np.float64) ** 2, axis=0))[::-1]
    assert cn[: len(cn) // 20].sum() > 0.5 * cn.sum()


def test_softmax_head_is_fixed():
    a, b = synth.softmax_head(64), synth.softmax_head(64)
    assert a.shape == (4, 64) and np.array_equal(a, b)
    assert abs(a.std() * np.sqrt(64) - 10.0) < 2.5
