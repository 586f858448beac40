"""Exact top-k context-sparse decode attention on MI355X (gfx950).

The HIP library (libsparse_decode.so) and its ctypes binding live in
``paper_2605_24168_amd.sparse_decode``; import that module to use the GPU
path.  ``paper_2605_24168_amd.synth`` draws seeded synthetic inputs.
"""
