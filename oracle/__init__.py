"""CPU oracle of the policy forward -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import anything here.  The GPU library never loads
it and it never loads the GPU library.
"""
