"""MI355X-native Jacobi-step engine (Jacobi Forcing, arXiv 2512.14681).

The hot path -- one Jacobi iteration: forward pass over the draft rows against
an exact paged KV cache, greedy vocabulary argmax, longest-prefix acceptance
and KV commit -- runs in hand-written HIP kernels for gfx950 behind the C ABI
of include/jf.h (libjf.so, built in-tree by ``build.py``).  ``jf`` is the
ctypes binding; ``decode`` holds the host-side decoding loops that drive it.
"""
