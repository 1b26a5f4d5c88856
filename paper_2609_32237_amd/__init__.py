"""MI355X-native batched FFT and SAR hot path (HIP kernels behind a C ABI).

``paper_2609_32237_amd._lib`` binds ``libmi355fft.so``; ``paper_2609_32237_amd.torch_api``
adds tensor conveniences on top of it (device pointers and streams only).
"""
