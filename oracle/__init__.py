"""CPU oracle for the VLM serving hot path (TEST INFRASTRUCTURE ONLY).

Plain, slow, float64 NumPy code that states what each stage computes, written from the
paper's definitions so that a reader can check it by eye:

* ``oracle.vlm``   -- vision encode, LLM prefill and paged LLM decode (Sec. 2.1, Sec. 2.2).
* ``oracle.sched`` -- the partition and scheduling formulas (Eq. 1-8, Alg. 1 policy).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  It shares no code with the HIP path and imports nothing from it;
the seeded input generators are passed in by the caller.  The product path never calls it.
"""
