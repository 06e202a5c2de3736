"""SPORK forked-decode hot path for MI355X (gfx950).

The compute path lives in ``libspork.so`` (hand-written HIP for CDNA4 behind a
C ABI declared in ``include/spork.h``); ``paper_2607_03333_amd.spork`` is its
thin Python binding. ``synth`` draws the seeded synthetic workloads.
"""
