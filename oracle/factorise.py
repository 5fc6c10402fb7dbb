"""Hybrid residual rank-1 SVD + magnitude pruning, float64 (oracle; test
infrastructure only).

Sec. III of the paper, "Hybrid compression and pruning" and Eq. (1): the
augmented matrix W_i = [W_x W_h] of each gate is approximated by a sum of
refinement steps.  Step n takes the top singular triplet (sigma, u, v) of the
current residual R^(n) = W_i - W~_i^(n-1), keeps only the NZ entries of v with
the largest magnitude ("prune(v, NZ)", the magnitude criterion of the
"Pruning by means of network sparsification" paragraph), and adds
sigma * u * prune(v)^T to the approximation.  Because each step is extracted
from the residual, the pruning error of earlier steps is corrected by later
ones.

Readings of points the paper leaves open (each is listed in the design notes):
  * groups: G=4 factorises each gate's H x C block separately (the paper's
    per-gate scheme); G=1 factorises the stacked 4H x C matrix;
  * pruning acts on v only (for a rank-1 term this is the same as keeping the
    NZ largest entries of every row, since row j is sigma*u_j*v^T); u is never
    pruned; sigma and u are not refit and v' is not renormalised;
  * magnitude ties go to the lower column index; masks are kept ascending;
  * sign: (u, v) is flipped so that the largest-magnitude entry of v (lowest
    index on ties) is positive;
  * a step whose sigma is <= 1e-12 * ||W_g||_2 ends the list: it and every
    later step are "terminated" (sigma = 0, u = 0, mask = {0..NZ-1}, value 0);
  * NZ = C - floor(p * C) for a pruning ratio p (p*C as one double product).
"""

from dataclasses import dataclass, field
import math

import numpy as np

STOP_REL = 1e-12


def nz_from_ratio(C, p):
    """Kept entries per v for pruning ratio p: C - floor(p*C), with p*C one
    IEEE double product (so any implementation doing the same gets the same NZ)."""
    return int(C - math.floor(float(p) * float(C)))


def top_triplet(R):
    """Top singular triplet (sigma, u, v) of R in float64.

    A left singular vector of R is an eigenvector of R R^T with eigenvalue
    sigma^2 (and a right one of R^T R); the eigensolver is LAPACK's symmetric
    one via ``numpy.linalg.eigh``.  The vector of the smaller Gram matrix is
    taken, and the other vector and sigma come from one product with R:
    v = R^T u / ||R^T u||, sigma = ||R^T u|| (or the transpose).
    Sign is left as the eigensolver returns it; ``prepare`` fixes it.
    """
    R = np.asarray(R, dtype=np.float64)
    m, n = R.shape
    if m <= n:
        w, Q = np.linalg.eigh(R @ R.T)
        u = Q[:, -1]
        r = R.T @ u
        sigma = float(np.linalg.norm(r))
        v = r / sigma if sigma > 0 else np.zeros(n)
        if sigma == 0:
            u = np.zeros(m)
    else:
        w, Q = np.linalg.eigh(R.T @ R)
        v = Q[:, -1]
        r = R @ v
        sigma = float(np.linalg.norm(r))
        u = r / sigma if sigma > 0 else np.zeros(m)
        if sigma == 0:
            v = np.zeros(n)
    return sigma, u, v


def fix_sign(u, v):
    """Flip (u, v) so that v's largest-magnitude entry (lowest index) is > 0."""
    k = int(np.argmax(np.abs(v)))          # argmax returns the first maximum
    if v[k] < 0:
        return -u, -v
    return u, v


def magnitude_mask(v, nz):
    """Indices of the nz entries of v with the largest |v|, ties to the lower
    index, returned ascending (Sec. III, magnitude-based pruning)."""
    v = np.asarray(v, dtype=np.float64)
    C = v.shape[0]
    order = np.lexsort((np.arange(C), -np.abs(v)))   # primary key: -|v|, then index
    return np.sort(order[:nz])


def round_bf16(a):
    """fp64 -> fp32 (round to nearest even) -> bf16 (round to nearest even),
    returned as float64 holding the bf16 value.  bf16 keeps the upper 16 bits
    of an IEEE binary32; rounding adds 0x7FFF plus the lowest kept bit before
    truncation (finite inputs only)."""
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


@dataclass
class Factors:
    """Refinement terms of every group, in extraction (= refinement) order."""
    D: int
    H: int
    groups: int
    rank: int
    nz: int
    sigma: np.ndarray      # [G][N]
    U: np.ndarray          # [G][N][R_g]
    mask: np.ndarray       # [G][N][NZ] int64, ascending
    vals: np.ndarray       # [G][N][NZ]  entries of prune(v) on the mask
    v_full: np.ndarray     # [G][N][C]   unpruned v (for certificates)
    eff_rank: np.ndarray   # [G]  live terms per group
    dtype: str = "f64"
    trajectory: list = field(default_factory=list)   # ||R^(n)||_F^2 per group

    @property
    def C(self):
        return self.D + self.H

    @property
    def rows(self):
        return 4 * self.H // self.groups

    def rounded(self, kind):
        """Copy with U and v' values stored as the library stores them:
        'f32' (fp64 -> fp32, nearest even) or 'bf16' (fp64 -> fp32 -> bf16).
        sigma is kept in fp32 in both cases.  Masks are unchanged: they are
        decided in fp64 before any rounding."""
        if kind == "f32":
            rnd = lambda a: np.asarray(a).astype(np.float32).astype(np.float64)
        elif kind == "bf16":
            rnd = round_bf16
        else:
            raise ValueError(kind)
        return Factors(self.D, self.H, self.groups, self.rank, self.nz,
                       self.sigma.astype(np.float32).astype(np.float64),
                       rnd(self.U), self.mask.copy(), rnd(self.vals),
                       self.v_full.copy(), self.eff_rank.copy(), kind,
                       list(self.trajectory))


def prepare(W, H, rank, nz, groups=4, record_trajectory=False, residual=True):
    """Factorise W = [W_ih | W_hh] ([4H, D+H], gate rows i, f, g, o) into
    ``rank`` pruned rank-1 refinement terms per group (Eq. (1)).

    For each group: R <- W_g; for n = 1..rank take the top triplet of R, fix
    its sign, keep the NZ largest-magnitude entries of v, store the term, and
    subtract sigma * u * prune(v)^T from R (the residual R^(n+1) = W - W~^(n)).

    residual=False is the alternative Sec. III contrasts the scheme with:
    successive higher-rank approximations of the original matrix, each term
    pruned on its own.  R then loses sigma * u * v^T with the unpruned v, so
    the terms are the singular triplets of W_g in order and the error that
    pruning leaves is never corrected by a later term.
    """
    W = np.asarray(W, dtype=np.float64)
    fourH, C = W.shape
    assert fourH == 4 * H and groups in (1, 4)
    D = C - H
    assert 1 <= nz <= C and rank >= 1
    Rg = fourH // groups
    sig = np.zeros((groups, rank))
    U = np.zeros((groups, rank, Rg))
    mask = np.tile(np.arange(nz, dtype=np.int64), (groups, rank, 1))
    vals = np.zeros((groups, rank, nz))
    vfull = np.zeros((groups, rank, C))
    eff = np.zeros(groups, dtype=np.int64)
    traj = []
    for g in range(groups):
        R = W[g * Rg:(g + 1) * Rg].copy()
        tr = [float(np.sum(R * R))] if record_trajectory else None
        tau = None
        live = 0
        for n in range(rank):
            s, u, v = top_triplet(R)
            if tau is None:
                tau = STOP_REL * s          # s at n = 0 is ||W_g||_2
            if s <= tau:
                break                        # this and every later term terminated
            u, v = fix_sign(u, v)
            m = magnitude_mask(v, nz)
            sig[g, n] = s
            U[g, n] = u
            mask[g, n] = m
            vals[g, n] = v[m]
            vfull[g, n] = v
            if residual:
                R[:, m] -= s * np.outer(u, v[m])
            else:
                R -= s * np.outer(u, v)
            live = n + 1
            if record_trajectory:
                tr.append(float(np.sum(R * R)))
        eff[g] = live
        traj.append(tr)
    return Factors(D, H, groups, rank, nz, sig, U, mask, vals, vfull, eff,
                   "f64", traj if record_trajectory else [])
