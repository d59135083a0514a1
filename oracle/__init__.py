"""CPU fp64 oracle for the CSR extend-attention path.

Test infrastructure only: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``.  The product library never
imports, links or calls anything here.
"""
