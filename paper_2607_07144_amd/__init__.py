"""MI355X-native hot path of the fractal KV-cache archive (arXiv 2607.07144).

The compute path is the C-ABI library ``libfkv.so`` (hand-written HIP kernels
for gfx950, sources under ``csrc/``), reached through the ctypes binding in
``paper_2607_07144_amd.fkv``.  Importing this package does not load the
library; importing ``paper_2607_07144_amd.fkv`` does, and fails loudly when it
is missing.
"""
__all__ = ["workloads"]
