"""MI355X-native batched simulation of distributed training strategies
(DistIR's simulator, Santhanam et al., MLSys 2022).

The simulation runs in the HIP kernels of ``libdsim.so`` behind the C ABI in
``include/dsim.h``; ``paper_2111_05426_amd.dsim`` is its Python binding,
``paper_2111_05426_amd.workloads`` holds the synthetic workload shapes,
``paper_2111_05426_amd.frontend`` binds the library's front end, which
turns programs written op by op into op tables (mixed abstract/concrete
interpretation, host C++), ``paper_2111_05426_amd.programs``
writes example programs for it, and ``paper_2111_05426_amd.calibrate`` fits the
empirical MatMul cost on the GPU it runs on.
"""
__all__ = ["dsim", "workloads", "frontend", "programs", "calibrate"]
