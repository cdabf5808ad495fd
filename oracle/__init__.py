"""CPU oracle for the synchronous data-parallel SGD step (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import this package.  It shares no code with the GPU library.
"""
