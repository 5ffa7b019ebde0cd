"""StepPrune inference-time selection on AMD MI355X (gfx950).

The HIP library (``libstepprune.so``, C ABI in ``include/stepprune.h``) runs
the paper's Algorithm 1: projection, the sequential pointer selection with
STOP, and the compaction of kept tokens.  ``binding`` is its thin ctypes
binding; ``workloads`` draws seeded synthetic inputs.  Importing this package
loads nothing; ``binding`` fails loudly when the library is missing.
"""
