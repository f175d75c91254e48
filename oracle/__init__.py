"""WnW CPU oracle: plain C in double precision, TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg may import
this package.  It shares no code with the HIP library and the two never import each other."""
