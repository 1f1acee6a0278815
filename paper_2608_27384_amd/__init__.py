"""MI355X (gfx950) streaming action decode for FlashVLA.

The compute path is libflashvla.so (hand-written HIP kernels behind the C ABI
of include/flashvla.h); ``paper_2608_27384_amd.flashvla`` is its ctypes
binding.  Importing this package does not load the library.
"""
