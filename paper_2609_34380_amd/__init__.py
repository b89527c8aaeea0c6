"""MI355X (gfx950) implementation of the nested-precision linear layer of
Dual-Mode Precision Serving: FP16 weights held as an FP8 upper-byte plane (E5M2,
or E4M3 for small-range layers) plus a chunked residual plane, contracted in
fast mode (upper plane only) or full mode (exact FP16 rebuilt in registers).

The compute lives in libdps.so (HIP kernels behind a C ABI, include/dps.h);
``paper_2609_34380_amd.dps`` is its thin Python binding.  Importing this
package does not load the library; the first call into ``dps`` does, and
fails loudly if it is not built.
"""

__all__ = ["dps", "graphs", "workloads"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module(__name__ + "." + name)
    raise AttributeError(name)
