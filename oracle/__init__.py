"""Float64 CPU oracle for the span-based tree CRF (test infrastructure).

This package is the slow, plain reference that the GPU path is checked
against. Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
CPU-baseline leg may import it; the product package never does, and the two
share no code (only the seeded input generators serve both).

Contents:
  crf_oracle.c   float64 inside / outside / reverse-mode / CKY / labelled CRF
  oracle.py      ctypes binding of that C library (numpy in, numpy out)
  bruteforce.py  enumeration of every binary bracketing, for tiny sentences
  build.py       compiles crf_oracle.c with gcc
"""
