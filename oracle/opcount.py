"""Operation counts and Table I arithmetic (oracle; test infrastructure only).

Sec. III: with the hybrid scheme the workload of each gate is
N_steps * (2R + 2NZ + 1) operations.  Sec. VI-B.1: the faithful (dense) gate
costs 2RC operations.  Table I reports latency per LSTM timestep, power and
performance efficiency in GOp/s/W; the efficiency column counts the
dense-equivalent work of the four gates, 4 * 2RC operations per timestep.
"""


def gate_ops_progressive(R, NZ, n_steps):
    return n_steps * (2 * R + 2 * NZ + 1)


def gate_ops_dense(R, C):
    return 2 * R * C


def table1_efficiency(latency_ms, power_w, R=64, C=8320):
    """GOp/s/W for one timestep of the 4-gate LSTM at the given latency."""
    ops = 4 * gate_ops_dense(R, C)
    return ops / (latency_ms * 1e-3) / power_w / 1e9
