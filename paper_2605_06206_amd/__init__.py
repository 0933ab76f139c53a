"""MI355X-native per-cluster MoE block of Federation of Experts.

The compute path is the hand-written HIP library ``libfoe.so`` (gfx950) behind a
C ABI (``include/foe.h``); ``paper_2605_06206_amd.foe`` is its thin Python
binding.  Importing this package loads nothing; the binding loads the library
on first use and raises if it has not been built.
"""

__all__ = ["foe", "synth", "build"]
