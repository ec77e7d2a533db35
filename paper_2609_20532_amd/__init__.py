"""MI355X (gfx950) DP-SGD gradient step: HIP kernels behind a C ABI.

Submodules: ``dpsgd`` (binding of ``include/dpsgd.h``), ``workloads`` (seeded
synthetic inputs), ``build`` (hipcc build of ``libdpsgd.so``). Importing the
package loads nothing; ``dpsgd.load()`` loads the library.
"""
