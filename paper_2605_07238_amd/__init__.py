"""MI355X-native horizon-aware candidate scoring (FATE, arXiv 2605.07238).

The scoring path runs in hand-written HIP kernels behind the C ABI declared in
``include/fate.h``; :mod:`paper_2605_07238_amd.fate` is the thin ctypes binding
and :mod:`paper_2605_07238_amd.synth` builds seeded synthetic workloads.
Nothing is imported eagerly, so the workload generator is usable without a GPU.
"""

__all__ = ["fate", "synth"]
