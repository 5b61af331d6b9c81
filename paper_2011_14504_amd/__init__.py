"""MI355X-native integer training kernels for the quantized dataflow of
arXiv 2011.14504 (int8 W/A/E/G convolutions, L1 batch normalization).

The compute lives in the HIP library libiseg.so (C ABI, include/iseg.h);
`paper_2011_14504_amd.iseg` is its thin Python binding.
"""
