"""Reference oracle for the activation-sparse FFN (test infrastructure, not product).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import anything under ``oracle/``.  It shares no code with the GPU library.
"""
