"""RhymeFlow keyframe-query attention path for AMD Instinct MI355X (gfx950).

The compute runs in ``librhymeflow.so`` (HIP kernels behind a C ABI, see
``include/rhymeflow.h``). ``paper_2606_06309_amd.binding`` is the thin Python
binding over that ABI; ``workloads`` draws seeded synthetic inputs and
``accounting`` holds the FLOP and byte counts used for rooflines.

Importing this package loads nothing native; importing ``binding`` does, and
raises if the HIP library has not been built.
"""
__version__ = "0.1.0"
