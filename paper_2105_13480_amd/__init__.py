"""MI355X-native (gfx950) CNN forward contraction.

Out[b,k,w,h] = sum_{c,r,s} In[b,c,sw*w+r,sh*h+s] * Ker[k,c,r,s]

The computation lives in hand-written HIP kernels behind the C ABI declared
in ``include/cnn.h`` (library ``libcnn_mi355x.so``).  ``paper_2105_13480_amd.cnn``
is the thin ctypes binding; ``paper_2105_13480_amd.inputs`` holds the seeded
synthetic workloads.  Submodules are imported lazily so that loading the
input generator never touches the GPU library.
"""

__all__ = ["cnn", "inputs"]
