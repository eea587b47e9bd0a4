"""MSA (MiniMax Sparse Attention) inference hot path for MI355X (gfx950).

Importing the package loads nothing; ``paper_2606_13392_amd.msa`` binds the
C-ABI library ``libmsa.so`` built from ``csrc/``.
"""
