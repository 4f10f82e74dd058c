"""MI355X (gfx950) replay of TRE's Token Service Share evaluation and
receiver/donor rebalancing.

``paper_2609_29160_amd.tre``     binding of the C ABI (include/tre.h)
``paper_2609_29160_amd.device``  uploading synthetic workloads to HBM
``paper_2609_29160_amd.build``   compiling libtre.so for gfx950
The binding is imported lazily so that building needs no GPU library.
"""
__all__ = ["tre", "device", "build"]
