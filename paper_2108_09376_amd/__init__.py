"""MI355X-native block-sparse convolution with temporal feature copying.

BlockCopy (Verelst & Tuytelaars, ICCV 2021) runs every convolution of a CNN only on
the image blocks a per-frame execution grid selects and keeps the previous
execution's features elsewhere (Section 3.1). This package is the hot path of that
method for AMD Instinct MI355X (gfx950):

* ``libblockcopy.so`` -- hand-written HIP kernels behind the C ABI of ``include/bc.h``
  (block index compaction, halo gather, block scatter, matrix-core sparse
  convolution with fused epilogue, sparse max pooling);
* :mod:`paper_2108_09376_amd.bc` -- the ctypes binding (same names as the C ABI);
* :mod:`paper_2108_09376_amd.resnet` -- a frame-by-frame ResNet-18/50 runner that
  keeps one persistent buffer per layer;
* :mod:`paper_2108_09376_amd.build` -- builds the library with hipcc for gfx950.

The binding raises at import if the library has not been built; there is no
fallback implementation.
"""
__all__ = ["bc", "resnet", "build"]
