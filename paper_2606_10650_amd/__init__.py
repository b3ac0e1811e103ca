"""MI355X (gfx950) implementation of the Dynamic Linear Attention layer forward
(arXiv 2606.10650): prefill and decode over a capacity-bounded state cache.

The HIP library (libdla.so) is loaded on first use by paper_2606_10650_amd.dla;
importing the package does not touch the GPU.
"""
__all__ = ["dla", "workloads", "build"]
