"""Float64 CPU oracle of the AMS image-embedding step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import, call or execute anything in
this package.  It shares no code with the HIP library it checks.
"""
