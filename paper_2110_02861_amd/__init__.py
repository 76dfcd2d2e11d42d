"""8-bit block-wise optimizers for MI355X (gfx950).

The fused 8-bit Adam / AdamW / Momentum step and standalone block-wise
quantize / dequantize of Dettmers et al., "8-bit Optimizers via Block-wise
Quantization", as hand-written HIP kernels behind the C-ABI library
``libbq.so`` (declared in ``include/bq.h``).  ``paper_2110_02861_amd.bq`` is the
thin ctypes binding over that library; PyTorch only supplies device memory and
streams.  ``paper_2110_02861_amd.workloads`` holds the seeded synthetic inputs.
"""
