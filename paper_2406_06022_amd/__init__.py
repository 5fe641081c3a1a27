"""MI355X-native relational graph-convolution (RGCN) block: forward and backward.

Submodules:
  rgcn   -- Python binding of the C-ABI library (librgcn.so): argument marshalling only.
  chain  -- multi-block mini-batch driver built on the binding.
  synth  -- seeded synthetic workloads (inputs only).
  build  -- compiles the HIP library for gfx950.
Importing the package loads nothing; ``rgcn`` loads the HIP library on first use and
raises if it is missing.
"""
__all__ = ["rgcn", "chain", "synth", "build"]
