"""MI355X-native mask-aware K/V-cached diffusion-transformer step (InstGenIE hot path).

``paper_2505_20600_amd.maskstep`` is the ctypes binding of the C ABI
(``include/maskstep.h``), ``paper_2505_20600_amd.workloads`` the seeded
synthetic workloads, ``paper_2505_20600_amd.build`` the in-tree hipcc build.
Nothing is imported eagerly, so importing the package never loads the GPU
library.
"""

__all__ = ["maskstep", "workloads", "build"]
