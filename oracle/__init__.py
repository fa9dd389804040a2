"""fp64 / exact-integer CPU oracle of the affinity path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this package.  It shares no code with the HIP library in
``paper_2609_13846_amd`` and imports nothing from it.
"""
