"""MI355X-native NVFP4 W4A4 linear layer (act-quant, weight prepack, GEMM with
per-segment global scales) behind a C ABI (``include/nvfp4.h``).

``paper_2609_04098_amd.nvfp4`` is the ctypes binding; it loads the HIP library
``libnvfp4.so`` built in this directory and fails loudly when it is missing.
``paper_2609_04098_amd.synth`` draws the seeded synthetic inputs.
"""
