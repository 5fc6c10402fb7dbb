"""Exact LSTM in float64 (oracle; test infrastructure only).

Sec. II and Fig. 1 of the paper: every gate takes the new input x^(t) and the
previous output h^(t-1) through W_x x + W_h h and a nonlinearity; the forget,
input and output gates use the logistic sigmoid and the cell gate uses tanh.
The cell state is c^(t) = f * c^(t-1) + i * c_hat and the output is
h^(t) = o * tanh(c^(t)).  No peepholes.

Readings (the paper is silent on these):
  * a bias b is added to the gate pre-activations, outside any approximation;
  * gate rows are stacked in the order i, f, g (cell candidate), o, so that
    ``torch.nn.LSTM`` (bias_ih = b, bias_hh = 0) computes the same function;
  * h0 = c0 = 0 unless given.
"""

import numpy as np


def sigmoid(z):
    """Logistic function 1/(1+exp(-z)), evaluated without overflow."""
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def cell_update(y, c_prev):
    """Gate nonlinearities and the c/h update of Sec. II.

    y: [..., 4H] pre-activations in row order i, f, g, o.  Returns (h, c).
    """
    y = np.asarray(y, dtype=np.float64)
    H = y.shape[-1] // 4
    i = sigmoid(y[..., 0 * H:1 * H])
    f = sigmoid(y[..., 1 * H:2 * H])
    g = np.tanh(y[..., 2 * H:3 * H])
    o = sigmoid(y[..., 3 * H:4 * H])
    c = f * c_prev + i * g
    h = o * np.tanh(c)
    return h, c


def exact_lstm(W, b, x, h0=None, c0=None):
    """Exact LSTM recurrence with the augmented matrix W = [W_x W_h].

    W: [4H, D+H]; b: [4H] or None; x: [T, B, D].
    Returns (h_seq [T, B, H], c_T [B, H]).
    Sec. III ("information-maximising approximation") defines the augmented
    matrix and the augmented input x~ = [x; h]; the gate products are the
    matrix-vector products of Fig. 1.
    """
    W = np.asarray(W, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    T, B, D = x.shape
    H = W.shape[0] // 4
    assert W.shape == (4 * H, D + H)
    bias = np.zeros(4 * H) if b is None else np.asarray(b, dtype=np.float64)
    h = np.zeros((B, H)) if h0 is None else np.asarray(h0, dtype=np.float64).copy()
    c = np.zeros((B, H)) if c0 is None else np.asarray(c0, dtype=np.float64).copy()
    hs = np.empty((T, B, H))
    for t in range(T):
        xt = np.concatenate([x[t], h], axis=1)          # [B, C]
        y = xt @ W.T + bias                              # [B, 4H]
        h, c = cell_update(y, c)
        hs[t] = h
    return hs, c


def row_tile_lstm(W, b, x, rows, h0=None, c0=None):
    """The dense baseline stopped part-way through each gate's rows.

    Sec. VI-B (comparison with the FPGA baseline): the faithful LSTM computes
    each gate's matrix-vector product in tiles of T_r rows, and the paper's
    baseline curve takes the LSTM output after every tile step.  Reading
    taken here: after ``rows`` rows of every gate (rows = m * T_r after m tile
    steps, the four gates advancing together as four parallel gate units),
    a computed row holds its full pre-activation b + W[row] . [x; h] and a row
    not reached yet holds the bias alone (so rows = 0 coincides with the
    progressive scheme at K = 0 and rows = H with the exact LSTM).  The same
    row budget applies at every timestep.

    W: [4H, D+H]; b: [4H] or None; x: [T, B, D]; 0 <= rows <= H.
    Returns (h_seq [T, B, H], c_T [B, H]).
    """
    W = np.asarray(W, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    T, B, D = x.shape
    H = W.shape[0] // 4
    assert W.shape == (4 * H, D + H) and 0 <= rows <= H
    bias = np.zeros(4 * H) if b is None else np.asarray(b, dtype=np.float64)
    h = np.zeros((B, H)) if h0 is None else np.asarray(h0, dtype=np.float64).copy()
    c = np.zeros((B, H)) if c0 is None else np.asarray(c0, dtype=np.float64).copy()
    hs = np.empty((T, B, H))
    for t in range(T):
        xt = np.concatenate([x[t], h], axis=1)          # [B, C]
        y = np.tile(bias, (B, 1))                        # [B, 4H]
        for q in range(4):                               # gates i, f, g, o
            for r in range(rows):
                o = q * H + r
                y[:, o] += xt @ W[o]
        h, c = cell_update(y, c)
        hs[t] = h
    return hs, c
