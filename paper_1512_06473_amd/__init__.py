"""PQ (product-quantized) layer forward of Q-CNN on AMD MI355X.

Paper: Wu et al., "Quantized Convolutional Neural Networks for Mobile
Devices", CVPR 2016.  The compute lives in libqcnn.so (HIP kernels for gfx950
behind the C ABI of include/qcnn.h); ``api`` is its Python binding.  Import
``paper_1512_06473_amd.api`` (needs the built library) or the pure-Python
helpers ``workloads`` and ``workmodel``.
"""
__all__ = ["api", "network", "workloads", "workmodel", "build"]
