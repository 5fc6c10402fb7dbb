"""Helpers shared by the GPU parity tests: run the library through the C ABI
binding and turn its exported terms into oracle Factors."""

import sys

import numpy as np
import torch

from oracle.factorise import Factors
from paper_1905_00689_amd import binding as B


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def rel_err(h_gpu, h_orc):
    """Max over (level, timestep, sequence) of ||h_gpu - h_orc||_inf / max(||h_orc||_inf, 1e-6)."""
    num = np.abs(h_gpu - h_orc).max(axis=-1)
    den = np.maximum(np.abs(h_orc).max(axis=-1), 1e-6)
    return float((num / den).max())


def prep(w, rank, p, groups=4, flags=0, factor_dtype=0):
    D, H = w.D, w.H
    return B.approx_lstm_prepare(w.W[:, :D], w.W[:, D:], w.b, D, H, rank, prune_ratio=p,
                                 groups=groups, flags=flags, factor_dtype=factor_dtype)


def run_gpu(m, x, levels, h0=None, c0=None, want_c=False, x_offset=0):
    """Run levels over x [T, B, D]; returns host (h [L, T, B, H], c [L, B, H] or None).
    x_offset > 0 places x that many floats into its device buffer (unaligned rows)."""
    T, Bn, D = x.shape
    H = m.info["hidden_size"]
    dev = torch.device("cuda")
    flat = np.ascontiguousarray(x, np.float32).reshape(-1)
    buf = torch.zeros(flat.size + x_offset, device=dev)
    buf[x_offset:] = torch.from_numpy(flat).to(dev)
    xt = buf[x_offset:].view(T, Bn, D)
    h_out = torch.full((len(levels), T, Bn, H), float("nan"), device=dev)
    c_out = torch.full((len(levels), Bn, H), float("nan"), device=dev) if want_c else None
    h0t = None if h0 is None else torch.from_numpy(np.ascontiguousarray(h0, np.float32)).to(dev)
    c0t = None if c0 is None else torch.from_numpy(np.ascontiguousarray(c0, np.float32)).to(dev)
    B.approx_lstm_run(m, xt, levels, h_out, h0t, c0t, c_out)
    B.approx_lstm_check(m)
    torch.cuda.synchronize()
    return h_out.cpu().numpy(), (c_out.cpu().numpy() if want_c else None)


def exported_factors(m):
    """The library's stored terms as an oracle Factors object (the stored
    values: fp32, or bf16 held exactly in fp32 for a bf16 model)."""
    inf = m.info
    G, N, Rg, nz, C = inf["groups"], inf["rank"], inf["rows_per_group"], inf["nz"], inf["aug_size"]
    sig = np.zeros((G, N)); U = np.zeros((G, N, Rg)); mask = np.zeros((G, N, nz), np.int64)
    vals = np.zeros((G, N, nz))
    for g in range(G):
        f = B.approx_lstm_get_factors(m, g)
        sig[g], U[g], mask[g], vals[g] = f["sigma"], f["u"], f["v_idx"], f["v_val"]
    kind = "bf16" if inf["factor_dtype"] == 1 else "f32"
    return Factors(inf["input_size"], inf["hidden_size"], G, N, nz, sig, U, mask, vals,
                   np.zeros((G, N, C)), np.array(inf["eff_rank"]), kind)
