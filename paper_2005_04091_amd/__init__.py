"""MI355X (gfx950) fused sparse direct convolution with CSR weights.

``paper_2005_04091_amd.spconv`` is the Python binding of the C-ABI library
``libspconv.so`` (declared in ``include/spconv.h``); importing it loads the library
and raises if it has not been built. ``paper_2005_04091_amd.synth`` draws the seeded
synthetic layers. Importing this package itself loads nothing.
"""
