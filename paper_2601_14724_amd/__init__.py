"""MI355X-native HERMES streaming step: chunk append with fused attention-mass
scoring, hierarchical-memory top-k eviction and order-preserving compaction.

The compute path is the C-ABI library ``libhermes.so`` (hand-written HIP for
gfx950); :mod:`paper_2601_14724_amd.hermes` is its thin Python binding and
:mod:`paper_2601_14724_amd.workloads` generates seeded synthetic inputs.
"""
__all__ = ["hermes", "workloads"]
