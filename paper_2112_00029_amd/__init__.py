"""MI355X (gfx950) hot path of Pixelated Butterfly: flat block butterfly +
low-rank linear layer (forward, backward-data, backward-weight) and
block-sparse attention, behind the C ABI of libpixelfly.so.

The binding is in `pixelfly`; importing it requires the built library
(`python -m paper_2112_00029_amd.build`).
"""
