"""Structurally sparsified LSTM backward pass on MI355X (gfx950).

Importing the package loads nothing; ``paper_1806_00512_amd.lstmss`` is the
binding to the native library and loads it on first use.
"""
