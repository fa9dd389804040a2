"""MI355X-native (gfx950) affinity-aware sharding for Delayed Tensor Parallelism.

``paper_2609_13846_amd.dtp`` is the ctypes binding of the C-ABI library ``libdtp.so``
(declared in ``include/dtp.h``); ``paper_2609_13846_amd.synth`` holds the seeded
synthetic inputs.  Importing the package loads nothing native.
"""
