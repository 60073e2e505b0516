"""MI355X-native QUASAR per-step loss-aware reconstruction.

The compute path is the HIP library ``libquasar.so`` (C ABI, ``include/quasar.h``);
``paper_2608_13966_amd.quasar`` is its thin ctypes binding and
``paper_2608_13966_amd.synth`` draws the seeded synthetic workloads.
Importing this package loads nothing; the library is opened on first use.
"""
__all__ = ["quasar", "synth"]
