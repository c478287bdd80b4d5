"""MI355X (gfx950) layer-wise prefix-KV reload and causal GQA prefill attention.

``swiftcache`` is the ctypes binding of the HIP library (``libswiftcache.so``,
built by ``build.py`` from ``csrc/``); ``workloads`` draws the seeded synthetic
inputs.  Importing the package loads neither torch nor the library.
"""
