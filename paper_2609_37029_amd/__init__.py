"""Fixed-cost speculative drafting (LongSpark's drafting step) on MI355X.

The computation lives in libldr.so (C ABI: include/ldr.h), built from the
HIP sources in csrc/ by ``python -m paper_2609_37029_amd.build``; the
binding is ``paper_2609_37029_amd.ldr``.
"""
