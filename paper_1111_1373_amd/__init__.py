"""MI355X (gfx950) evaluation of classification trees: data and speculative decompositions.

The compute path is the C-ABI library ``libdtree.so`` (hand-written HIP kernels); the
Python module ``paper_1111_1373_amd.dtree`` binds it.  Import that module explicitly; this
package file loads nothing so that the seeded workload generators can be imported on
machines without the library.
"""
__all__ = ["dtree", "workloads"]
