"""Seeded synthetic workloads for the progressive approximate-LSTM path.

This module is the one piece shared by the product's tests/bench and the CPU
oracle: it only draws random numbers (no part of the method's arithmetic).

The paper's driving workload (Sec. VI-A: FCN features of dashcam frames fed to
an LSTM; neither the videos nor the trained weights are available) is stood in
for by Gaussian weights with standard deviation 1/sqrt(D+H), Gaussian biases
with standard deviation 0.1, and ReLU-like inputs max(0, N(0,1)) (about half
exact zeros), the shape of CNN feature maps after a rectifier.

Every workload draws, from ``numpy.random.default_rng([190500689, index])``,
the weight matrix W = [W_ih | W_hh] as one [4H, D+H] row-major matrix, then
the bias b [4H], then the inputs x [T, B, D] (layer by layer for stacks), in
float64, and casts them to float32.  Gate rows are ordered i, f, g, o.
"""

from dataclasses import dataclass, field

import numpy as np

SEED = 190500689


def rng_for(index):
    return np.random.default_rng([SEED, int(index)])


def lstm_weights(rng, D, H):
    """(W [4H, D+H] fp32, b [4H] fp32) with W ~ N(0, sd 1/sqrt(D+H)), b ~ N(0, sd 0.1)."""
    C = D + H
    W = rng.normal(0.0, 1.0 / np.sqrt(C), size=(4 * H, C)).astype(np.float32)
    b = rng.normal(0.0, 0.1, size=(4 * H,)).astype(np.float32)
    return W, b


def lstm_weights_decay(rng, D, H, alpha=1.0, beta=1.0):
    """(W [4H, D+H] fp32, b [4H] fp32) with decaying spectra and decaying
    column importance: the redundancy a trained LSTM shows and the Gaussian
    model (flat spectrum, every input equally weighted) lacks.

    Column k of every gate block is scaled by c_k = (pi(k)+1)^-beta for one
    random permutation pi of the D+H columns (a few inputs carry most of the
    weight, as for CNN features); each gate block is then
    Q_u diag(s) Q_v^T diag(c) with Q_u [H, H] and Q_v [D+H, H] orthonormal
    (QR of Gaussian matrices, signs fixed by the diagonal of R) and
    s_i = (i+1)^-alpha, rescaled so that the block's squared Frobenius norm
    is H, as for the Gaussian model.  Bias as in lstm_weights."""
    C = D + H
    c = np.empty(C)
    c[rng.permutation(C)] = (np.arange(C) + 1.0) ** (-beta)
    blocks = []
    for _ in range(4):
        qu, ru = np.linalg.qr(rng.normal(size=(H, H)))
        qu *= np.sign(np.diag(ru))
        qv, rv = np.linalg.qr(rng.normal(size=(C, H)))
        qv *= np.sign(np.diag(rv))
        sv = (np.arange(H) + 1.0) ** (-alpha)
        blk = ((qu * sv) @ qv.T) * c
        blocks.append(blk * np.sqrt(H / np.sum(blk * blk)))
    W = np.concatenate(blocks, axis=0).astype(np.float32)
    b = rng.normal(0.0, 0.1, size=(4 * H,)).astype(np.float32)
    return W, b


def features(rng, T, B, D, kind):
    """Inputs x [T, B, D] fp32: 'normal' N(0,1) or 'relu' max(0, N(0,1))."""
    x = rng.normal(0.0, 1.0, size=(T, B, D))
    if kind == "relu":
        x = np.maximum(x, 0.0)
    elif kind != "normal":
        raise ValueError(kind)
    return x.astype(np.float32)


@dataclass
class Workload:
    name: str
    D: int
    H: int
    T: int
    B: int
    layers: list = field(default_factory=list)     # [(W, b)] per layer
    x: np.ndarray = None

    @property
    def W(self):
        return self.layers[0][0]

    @property
    def b(self):
        return self.layers[0][1]


def make(D, H, T, B, index, xkind="relu", n_layers=1, name="custom", wkind="gaussian"):
    """Generic seeded workload: n_layers LSTM layers (D -> H -> H ...), then x.
    wkind 'gaussian' (lstm_weights) or 'decay' (lstm_weights_decay)."""
    rng = rng_for(index)
    layers = []
    d = D
    for _ in range(n_layers):
        if wkind == "gaussian":
            layers.append(lstm_weights(rng, d, H))
        elif wkind == "decay":
            layers.append(lstm_weights_decay(rng, d, H))
        else:
            raise ValueError(wkind)
        d = H
    x = features(rng, T, B, D, xkind)
    return Workload(name, D, H, T, B, layers, x)


def softmax_head(H, n_out=4, index=0):
    """A fixed random read-out [n_out, H] fp32 (N(0, sd 10/sqrt(H))) that turns
    each h into n_out logits: a stand-in for the driving model's 4-way
    prediction layer, used only to express output error as the KL divergence
    between class distributions.  The scale keeps the predictions away from
    uniform for h with entries of a tenth or two (top class probability about
    0.45-0.65 on average on the named workloads)."""
    rng = np.random.default_rng([SEED, 1000 + int(index)])
    return rng.normal(0.0, 10.0 / np.sqrt(H), size=(n_out, H)).astype(np.float32)


# The named workloads and their parameters.
TINY = dict(D=64, H=32, T=8, B=1, index=1, xkind="normal", name="tiny")
DRIVING = dict(D=2048, H=512, T=16, B=1, index=2, xkind="relu", name="driving")
BATCHED = dict(D=2048, H=512, T=16, B=256, index=2, xkind="relu", name="batched")
STACK = dict(D=4096, H=1024, T=32, B=1, index=4, xkind="relu", n_layers=2, name="stack")
DEADLINE = dict(D=2048, H=2048, T=64, B=8, index=5, xkind="relu", name="deadline")
# The paper's own model shape (Sec. VI-A: 8256 FCN features into 64 hidden
# units, 100-frame sequences) with decaying-spectrum weights.
PAPER = dict(D=8256, H=64, T=100, B=1, index=6, xkind="relu", wkind="decay", name="paper")
# The driving shape with decaying-spectrum weights.
DRIVING_DECAY = dict(D=2048, H=512, T=16, B=1, index=7, xkind="relu", wkind="decay", name="driving-decay")
# The deadline shape with decaying-spectrum weights.
DEADLINE_DECAY = dict(D=2048, H=2048, T=64, B=8, index=8, xkind="relu", wkind="decay", name="deadline-decay")

NAMED = {w["name"]: w for w in (TINY, DRIVING, BATCHED, STACK, DEADLINE, PAPER, DRIVING_DECAY, DEADLINE_DECAY)}


def named(name, **override):
    kw = dict(NAMED[name])
    kw.update(override)
    return make(**kw)
