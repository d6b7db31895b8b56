"""CPU oracle for the fused matmul + bias + ReLU (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never does.
"""
