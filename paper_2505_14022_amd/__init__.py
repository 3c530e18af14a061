"""libmsda: multi-scale deformable attention (MSDA) forward and backward for AMD MI355X (gfx950).

The compute path is the C-ABI library ``libmsda.so`` (hand-written HIP kernels); the Python
module :mod:`paper_2505_14022_amd.msda` is a thin ctypes binding over it. Importing this
package loads nothing; the library is loaded on first use and a missing library is an error.
"""

__all__ = ["msda", "workloads"]
