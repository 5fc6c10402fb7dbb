"""The measurement arithmetic of bench.py on the CPU: the algorithmic bytes
and flops per timestep that the roofline fractions divide by.

Per timestep the method streams, for each of the G*K refinement terms in use
(Eq. (1)), u (4 R_g bytes), v's kept entries (NZ fp32 values and 16-bit
column indices, or the dense fp32 vector when nothing is pruned) and sigma,
plus x_t and the h outputs; the paper counts N_steps (2R + 2NZ + 1) operations
per gate (Sec. III).  The expected values below are those sums worked out by
hand for the workloads the bench times.
"""

import bench


def test_driving_bytes_per_timestep():
    # 4 gates x 512 terms x (2048 + 3840 + 4) + x (8192) + h (2048)
    assert bench.algorithmic_bytes_per_timestep(4, 512, 640, 2560, 512, 2048, 512, 1, 1) == 12_077_056
    # no pruning: v streamed dense, 4 x 2560 bytes per term
    assert bench.algorithmic_bytes_per_timestep(4, 512, 2560, 2560, 512, 2048, 512, 1, 1) == 25_184_256
    # K = 0 leaves x and h only
    assert bench.algorithmic_bytes_per_timestep(4, 512, 640, 2560, 0, 2048, 512, 1, 1) == 10_240


def test_deadline_and_stack_bytes_per_timestep():
    # D = H = 2048, 8 sequences, rank 2048, NZ = 410: 8192 terms x 10656 + 2 x 65536
    assert bench.algorithmic_bytes_per_timestep(4, 2048, 410, 4096, 2048, 2048, 2048, 8, 1) == 87_425_024
    # stacked layers at (1024, 1024): 4096 x 11780 + 20480, then 4096 x 7172 + 8192
    assert bench.algorithmic_bytes_per_timestep(4, 1024, 1280, 5120, 1024, 4096, 1024, 1, 1) == 48_271_360
    assert bench.algorithmic_bytes_per_timestep(4, 1024, 512, 2048, 1024, 1024, 1024, 1, 1) == 29_384_704


def test_paper_operation_count():
    # 4 gates x 512 steps x (2 x 512 + 2 x 640 + 1)
    assert bench.algorithmic_flops_per_timestep(4, 512, 640, 512, 1) == 4_720_640
    assert bench.algorithmic_flops_per_timestep(4, 512, 640, 512, 256) == 256 * 4_720_640


def test_batched_mfma_flops():
    # x-projection 2 x 2048 rows x 2048 x 16 timesteps x 256 sequences, then per
    # timestep the h-projection (2 x 2048 x 512 x 256) and the accumulation
    # (2 x 2048 rows x 512 terms x 256)
    assert bench.mfma_flops_batched(4, 2048, 512, 16, 256, 512) == 51_539_607_552
    # budgets and sizes are padded to the 32-wide contraction: K = 20 runs as 32
    assert bench.mfma_flops_batched(4, 2048, 512, 16, 256, 20) == bench.mfma_flops_batched(4, 2048, 512, 16, 256, 32)
