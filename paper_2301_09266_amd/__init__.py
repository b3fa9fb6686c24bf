"""FInC Flow masked k x k convolution on MI355X (gfx950).

The compute lives in the HIP library `csrc/libfinc.so` behind the C ABI of
`include/finc.h`; `finc` is its thin Python binding (argument marshalling
only, PyTorch for device memory and streams).
"""
