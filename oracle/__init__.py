"""fp64 CPU oracle for prefix-reuse attention.

TEST INFRASTRUCTURE ONLY: imported by the test suite, by the package smoke
check and by the benchmark's CPU-baseline leg, never by the GPU product path.
It shares no code with the GPU library.

* ``kvr_ref.c`` / ``ref.py`` -- threaded fp64 attention (prefill, continue,
  cache append), the checker for every GPU parity test.
* ``brute.py``              -- pure-Python triple loop that pins the compiled
  oracle on tiny shapes.
"""
