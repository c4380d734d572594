"""BAG budget-aware cached DiT sampling on MI355X (gfx950).

The package is deliberately lazy: importing it does not load the HIP
library.  ``paper_2608_09231_amd.binding`` loads ``libdit_cache.so`` and
raises if it is missing; ``paper_2608_09231_amd.synth`` holds the seeded
input generators and the workload registry and touches no GPU code.
"""

__all__ = ["binding", "synth", "build"]
