"""libkgq: batched complex-logical-query answering on AMD Instinct MI355X.

The compute path lives in the HIP library ``libkgq.so`` built from
``csrc/``; :mod:`paper_2503_02172_amd.kgq` is its ctypes binding and
:mod:`paper_2503_02172_amd.synth` draws the seeded synthetic workloads.
Importing this package loads nothing; the library is opened on first use.
"""
