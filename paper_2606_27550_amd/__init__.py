"""EntMTP tree-verification hot path for AMD Instinct MI355X (gfx950).

The compute path lives in ``libentmtp.so`` (HIP kernels behind a C ABI, see
``include/entmtp.h``); :mod:`paper_2606_27550_amd.api` is a thin ctypes binding
that only marshals arguments.  :mod:`paper_2606_27550_amd.synth` draws the
seeded synthetic workloads.
"""
