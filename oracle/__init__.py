"""CPU oracle for the N-MDLM block-denoising step.  Test infrastructure only:
imported by ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py``; the HIP library never calls it."""
