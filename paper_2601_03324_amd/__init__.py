"""MI355X-native (gfx950) TVL GEMV: the per-token weight sweep y = W x of a
Llama-2 decode step (Kilictas & Alpay, arXiv 2601.03324) as a C-ABI HIP
library.  ``tvl`` is the Python binding of that library."""
__all__ = ["tvl", "build"]
