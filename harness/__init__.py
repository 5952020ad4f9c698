"""Benchmark and test harness: seeded synthetic inputs and work accounting.

Shared by the tests, the benchmark and the smoke check.  It holds none of the
attention arithmetic: the GPU path lives in ``paper_2606_13361_amd`` and the
fp64 checker in ``oracle``.
"""
