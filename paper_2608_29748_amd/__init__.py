"""MI355X-native ReTrace speculative-decoding round (HIP kernels behind a C ABI).

`binding` exposes the C ABI of include/retrace.h; `engine` owns device memory
(PyTorch tensors) around it.
"""
