"""MI355X-native mini-batch training of fully connected feed-forward networks
(the data-parallel hot path of neural-fortran, arXiv:1902.06714).

The compute runs in hand-written HIP kernels behind the C ABI declared in
``include/nf.h``; ``paper_1902_06714_amd.nf`` is the thin ctypes binding.
"""
