"""MI355X-native mixed-precision MoE block (MxMoE, arXiv 2505.05799).

The compute path lives in ``libmxmoe.so`` (HIP kernels for gfx950 behind the
C ABI declared in ``include/mxmoe.h``).  ``paper_2505_05799_amd.mxmoe`` is the
thin ctypes binding; ``paper_2505_05799_amd.workloads`` holds the seeded
synthetic inputs.  Importing this package loads neither.
"""

__all__ = ["mxmoe", "workloads"]
