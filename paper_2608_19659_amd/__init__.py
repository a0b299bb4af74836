"""libfleetsieve: an MI355X-native (gfx950) implementation of FleetSieve's
decision-critical acquisition scorer.

The compute lives in ``libfleetsieve.so`` (hand-written HIP kernels behind a
C ABI, declared in ``include/fleetsieve.h``).  ``paper_2608_19659_amd.fleetsieve``
is the thin ctypes binding; ``paper_2608_19659_amd.synth`` draws seeded
synthetic workloads.  Importing the package loads nothing: the binding loads
the library on first use and raises if it is missing.
"""
__all__ = ["fleetsieve", "synth"]
