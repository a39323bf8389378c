"""kvx: paged KV-cache gather / scatter / transfer for MI355X (gfx950).

The copy engine is a C-ABI library (``libkvx.so``) of hand-written HIP
kernels; ``paper_2606_31093_amd.kvx`` is its thin Python binding and
``paper_2606_31093_amd.workloads`` generates seeded synthetic inputs.
"""
