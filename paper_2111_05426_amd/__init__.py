"""MI355X-native batched simulation of distributed training strategies
(DistIR's simulator, Santhanam et al., MLSys 2022).

The simulation runs in the HIP kernels of ``libdsim.so`` behind the C ABI in
``include/dsim.h``; ``paper_2111_05426_amd.dsim`` is its Python binding and
``paper_2111_05426_amd.workloads`` holds the synthetic workload shapes.
"""
__all__ = ["dsim", "workloads"]
