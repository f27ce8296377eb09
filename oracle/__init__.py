"""CPU oracle for batched pipeline-schedule simulation — test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may load it.
"""
