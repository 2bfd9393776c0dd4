"""Continual convolution and pooling steps on AMD MI355X (gfx950).

The compute path is the C-ABI library ``libcoinf.so`` (hand-written HIP
kernels); ``paper_2204_03418_amd.coinf`` is its thin ctypes binding and
``paper_2204_03418_amd.synth`` holds the seeded synthetic inputs.  Importing
the package itself loads nothing; importing ``coinf`` loads the library and
raises if it has not been built.
"""
