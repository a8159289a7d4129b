"""MI355X-native two-tier KV-cache decode path of CMC (Context-to-Answer-
Aligned Memory Compression): question-guided Tier-1 top-k selection of
context memory embeddings and decode attention over the selected memory
rows plus a Tier-2 local-window ring buffer (Sec. 2.5 of the paper).

The compute runs in hand-written HIP kernels for gfx950 behind the C ABI in
``include/cmc.h`` (``libcmc.so``); ``paper_2609_25537_amd.cmc`` is the thin
Python binding over it.  Importing this package loads nothing; the binding
loads the library on first use and raises if it is missing.
"""
