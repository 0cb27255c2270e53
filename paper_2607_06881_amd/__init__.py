"""Multiple-double matrix product C = A·B on one MI355X (gfx950).

The product of two multiple-double matrices (double-double, triple-double or
quad-double) is computed by splitting every operand exactly into 13-bit integer
slices on a shared power-of-two grid per row of A and per column of B, running
the slice pairs as exact FP64 GEMMs on the matrix cores, and recombining the
level products exactly (Chen and Verschelde, "Multiple Double Arithmetic on
NVIDIA Tensor Cores", sections 2 and 3).

Submodules are imported lazily so that the input generator can be used without
loading the HIP library:

* ``paper_2607_06881_amd.workloads`` - seeded synthetic operands (numpy only).
* ``paper_2607_06881_amd.mdgemm``    - ctypes binding of ``libmdgemm.so``.
* ``paper_2607_06881_amd.build``     - compiles ``libmdgemm.so`` for gfx950.
"""

__all__ = ["workloads", "mdgemm", "build"]


def __getattr__(name):
    if name in __all__:
        import importlib

        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
