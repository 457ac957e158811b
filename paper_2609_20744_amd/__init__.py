"""Video Delta Attention (VDA) forward pass for MI355X (gfx950).

The compute path lives in the HIP library ``libvda.so`` (C ABI declared in
``include/vda.h``); :mod:`paper_2609_20744_amd.vda` is its thin ctypes binding.
:mod:`paper_2609_20744_amd.inputs` generates seeded synthetic workloads.
"""
