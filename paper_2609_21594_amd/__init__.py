"""MI355X-native batched Muon step: HIP kernels for gfx950 behind a C ABI.

The compute path lives in ``csrc/`` (built into ``libmuon_hip.so``); the
``binding`` module marshals torch tensors to that library, and ``optim``
wraps it as a torch optimizer (Muon for matrices, chained AdamW for the
rest).  ``synth`` holds the seeded synthetic workloads.  Importing the package loads nothing native;
the binding loads the library on first use and raises if it is missing.
"""
__all__ = ["binding", "optim", "synth"]
