"""MI355X-native block-memory attention step of InfLLM (arXiv 2402.04617).

The compute lives in libinfllm.so (hand-written HIP for gfx950, C ABI in
include/infllm.h); `paper_2402_04617_amd.infllm` is its ctypes binding.
Importing this package does not load the library; the first call does, and
fails loudly if it has not been built.
"""
