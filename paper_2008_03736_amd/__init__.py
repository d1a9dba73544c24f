"""MI355X (gfx950) batched tree-CRF inside / marginals / CKY.

The compute path is the HIP library ``libcrfinside.so`` (C ABI declared in
``include/crf_inside.h``); ``binding`` marshals arguments to it.  Importing
this package does not load the library: ``binding.load()`` does, and raises if
it is missing.  ``workloads`` holds the seeded synthetic input generators.
"""
__all__ = ["binding", "workloads"]
