"""MI355X-native hot path of MORI's idleness-ranked KV tier placement
(arXiv 2606.00866): a C-ABI library of gfx950 HIP kernels (libmori.so) and a
thin Python binding.  ``mori`` holds the binding, ``tiering`` a small
caller-side runtime (device state tensors, pinned CPU-tier arena)."""
