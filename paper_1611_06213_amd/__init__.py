"""GaDei-style ASGD parameter server on one gfx950 GPU.

The server's hot path (push -> fused K-gradient apply -> pull fan-out) lives
in the HIP library built from csrc/ (libgadeips.so); `ps` is its thin ctypes
binding and `workloads` the seeded synthetic inputs. Importing the package
loads nothing: the binding loads the library on first use and raises if it
is not built.
"""
