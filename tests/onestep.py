"""One-step parity of a factor chain: for every checked step n, rebuild the
residual R^(n) = W_g - sum_{m<n} sigma_m u_m prune(v_m)^T from the chain's own
float64 terms and let the oracle take that step (top triplet, sign, mask).
Test helper; uses only oracle/ for the arithmetic it checks against."""

import numpy as np

import oracle
from oracle.factorise import fix_sign


def residual_before(Wg, sig, U, V, masks, n):
    R = np.array(Wg, dtype=np.float64, copy=True)
    for m in range(n):
        k = masks[m]
        R[:, k] -= sig[m] * np.outer(U[m], V[m][k])
    return R


def check_steps(Wg, sig, U, V, masks, nz, steps, gap_floor=1e-9, progress=None):
    """Returns a list of (n, status) with status 'exact' (masks equal) or
    'tie' (mask threshold gap below gap_floor, either mask acceptable).
    Raises AssertionError on a real disagreement.  progress(n), if given, is
    called after each checked step."""
    out = []
    steps = sorted(steps)
    R = np.array(Wg, dtype=np.float64, copy=True)
    done = 0
    for n in steps:
        for m in range(done, n):
            k = masks[m]
            R[:, k] -= sig[m] * np.outer(U[m], V[m][k])
        done = n
        s, u, v = oracle.top_triplet(R)
        u, v = fix_sign(u, v)
        assert abs(s - sig[n]) <= 1e-10 * s, (n, s, sig[n])
        assert np.linalg.norm(v - V[n]) <= 1e-8, (n, np.linalg.norm(v - V[n]))
        assert np.linalg.norm(u - U[n]) <= 1e-8, (n, np.linalg.norm(u - U[n]))
        m_orc = oracle.magnitude_mask(v, nz)
        if np.array_equal(m_orc, masks[n]):
            out.append((n, "exact"))
        else:
            a = np.sort(np.abs(v))[::-1]
            gap = (a[nz - 1] - a[nz]) / a[nz - 1] if nz < len(a) else 1.0
            assert gap < gap_floor, (n, gap)
            out.append((n, "tie"))
        if progress:
            progress(n)
    return out
