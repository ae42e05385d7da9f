"""Graph-segment decode attention for GraphPO rollouts on MI355X (gfx950).

The compute path lives in the HIP library ``libgraphattn.so`` behind a C ABI
(``include/graphattn.h``); ``paper_2606_18954_amd.graphattn`` is its thin ctypes binding.
``paper_2606_18954_amd.workloads`` draws seeded synthetic rollout graphs.
"""
__all__ = ["graphattn", "workloads"]
