"""CPU oracle for the Winograd 3x3 convolution (test infrastructure only).

This package is the correctness reference for the GPU library.  It is plain,
slow and meant to be checked against the paper by eye:

* ``direct``      -- Eq. 1 of the paper (the layer definition) as a plain C
                     direct convolution with fp64 accumulation (``direct_conv.c``).
* ``toom_cook``   -- exact rational Winograd/Toom-Cook transform matrices
                     (the paper's A, B, G of Eq. 3, which it does not print).
* ``winograd``    -- an fp64 NumPy Winograd F(m x m, 3 x 3) following Eq. 3 and
                     the overlap-add tiling of Sec. 2.1, exposing the
                     intermediates of the three steps of Sec. 3.
* ``shared_buffer`` -- the shared-buffer size and overwrite rule of Sec. 4.2.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call, link or execute anything in this package.  The
GPU library never does, and this package imports nothing from it: the two share
no code, tables or generators.
"""
