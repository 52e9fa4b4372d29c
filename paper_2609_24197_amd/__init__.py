"""MI355X (gfx950) implementation of H-Spec's block-parallel drafting step.

``hspec`` is the ctypes binding of the HIP library ``libhspec.so``;
``inputs`` holds the seeded synthetic workload generators.
"""
