"""FlexMoE masked MoE-layer forward for MI355X (gfx950).

The compute path is the HIP library ``libflexmoe.so`` built from ``csrc/``;
``flexmoe`` holds its thin ctypes binding.  ``synth`` holds the seeded input
generators.  Importing the package loads nothing native: the binding loads the
library on first use and raises if it is missing.
"""
__all__ = ["synth", "flexmoe"]
