"""CPU oracle for the multiple-double matrix product -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import, call, link or execute anything in this package.  The
GPU product path never does, and the two share no code.

* ``exact``   -- plain definitions in Python integers and fractions (slow, exact).
* ``coracle`` -- the C oracle: error-free transformations, classic
  multiple-double arithmetic and GEMM (the timed CPU baseline), the exact
  big-integer splitter and int64 slice products.
* ``pipeline`` -- the method's steps chained on the CPU for sampled entries.
"""
