"""Error-feedback gradient sparsification for MI355X (gfx950).

The compression step of "Rethinking gradient sparsification as total error
minimization" (arXiv 2108.00951): the hard-threshold sparsifier with error
feedback, the Top-k baseline, and the sparse exchange-and-average of n
workers' payloads.  All arithmetic runs in hand-written HIP kernels behind
the C ABI of ``libefsparse.so``; this package only marshals arguments.
"""
__all__ = ["binding", "synth"]
