"""MI355X-native progressive approximate-LSTM inference (arXiv 1905.00689).

The compute path lives in ``libapprox_lstm.so`` (hand-written HIP kernels for
gfx950 behind a C ABI declared in ``include/approx_lstm.h``);
``paper_1905_00689_amd.binding`` marshals arguments to it and
``paper_1905_00689_amd.synth`` draws the seeded synthetic workloads.  Import
the submodule you need; this package file loads nothing by itself.
"""
