"""Progressive gate evaluation under a refinement budget, float64 (oracle;
test infrastructure only).

Eq. (1) of the paper: the approximate pre-activation of gate i after
N_steps refinement steps is the sum over n of
sigma^(n) * u^(n) * (prune(v^(n), NZ)^T x~), with x~ = [x^(t); h^(t-1)] the
augmented input of Sec. III.  Each step is a dot product, a scaling by sigma
and an accumulation into the gate output (the 2R + 2NZ + 1 operations per step
stated after Eq. (1)).  The gate outputs then go through the cell update of
Sec. II.

Readings: the bias is added exactly; budget K counts refinement steps per group
(the paper's N_steps); terminated terms contribute nothing; each requested
level K_j is its own recurrence over the whole sequence (the paper evaluates
each (NZ, N_steps) design as a separate approximate LSTM); ``run_schedule``
takes one K per timestep (a deadline run replayed).
"""

import numpy as np

from .lstm import cell_update
from .factorise import round_bf16


def dense_pruned_v(f, g):
    """prune(v^(n)) of group g for every n, as dense [N][C] rows (zeros off the mask)."""
    V = np.zeros((f.rank, f.C))
    rows = np.arange(f.rank)[:, None]
    V[rows, f.mask[g]] = f.vals[g]
    return V


def reconstruct(f, g, K):
    """W~_g^(K) = sum_{n<=K} sigma_n u_n prune(v_n)^T  (the approximation after K steps)."""
    V = dense_pruned_v(f, g)
    K = min(K, f.rank)
    return (f.U[g, :K].T * f.sigma[g, :K]) @ V[:K]


def run_schedule(f, b, x, Ks, h0=None, c0=None, operand_round=None):
    """One recurrence with budget Ks[t] at timestep t.

    f: Factors; b: [4H] or None; x: [T, B, D].  Returns (h [T, B, H], c_T [B, H]).
    operand_round='bf16' gives both products bf16 operands, as the batched
    bf16 configuration computes them (bf16 operands, fp32 accumulation):
    x~ is rounded before prune(v)^T x~, and z = sigma * s before the
    accumulation into the gates (the factor values come rounded in f).
    """
    x = np.asarray(x, dtype=np.float64)
    T, B, D = x.shape
    H, G, Rg = f.H, f.groups, f.rows
    assert D == f.D and len(Ks) == T
    bias = np.zeros(4 * H) if b is None else np.asarray(b, dtype=np.float64)
    Vd = [dense_pruned_v(f, g) for g in range(G)]
    h = np.zeros((B, H)) if h0 is None else np.asarray(h0, dtype=np.float64).copy()
    c = np.zeros((B, H)) if c0 is None else np.asarray(c0, dtype=np.float64).copy()
    hs = np.empty((T, B, H))
    for t in range(T):
        xt = np.concatenate([x[t], h], axis=1)            # x~ for every sequence, [B, C]
        if operand_round == "bf16":
            xt = round_bf16(xt)
        y = np.zeros((B, 4 * H))
        for g in range(G):
            n = int(min(Ks[t], f.eff_rank[g]))
            if n <= 0:
                continue
            s = Vd[g][:n] @ xt.T                          # prune(v_n)^T x~   [n, B]
            z = f.sigma[g, :n, None] * s                  # sigma_n * s_n
            if operand_round == "bf16":
                z = round_bf16(z)
            y[:, g * Rg:(g + 1) * Rg] += (f.U[g, :n].T @ z).T   # sum_n z_n u_n
        y += bias
        h, c = cell_update(y, c)
        hs[t] = h
    return hs, c


def run(f, b, x, levels, h0=None, c0=None, operand_round=None):
    """Independent recurrences at each budget in ``levels``.

    Returns (h [L, T, B, H], c [L, B, H]).
    """
    x = np.asarray(x, dtype=np.float64)
    T, B, _ = x.shape
    L = len(levels)
    hs = np.empty((L, T, B, f.H))
    cs = np.empty((L, B, f.H))
    for j, K in enumerate(levels):
        hs[j], cs[j] = run_schedule(f, b, x, [K] * T, h0, c0, operand_round)
    return hs, cs
