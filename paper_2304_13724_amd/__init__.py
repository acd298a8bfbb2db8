"""MI355X-native blocked SGD matrix factorisation (BGMF).

The compute path is the HIP library ``libbgmf.so`` (sources in ``csrc/``,
C ABI in ``include/bgmf.h``); ``bgmf`` is its ctypes binding.  Importing
``paper_2304_13724_amd.bgmf`` fails if the library has not been built.
"""
