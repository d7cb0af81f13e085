"""ResBM residual bottleneck boundary module on MI355X (gfx950).

Importing the package loads nothing native; ``paper_2604_11947_amd.resbm``
binds the C-ABI library ``libresbm.so`` on first use.
"""
