"""MI355X-native fused RoPE + masked attention (AttnFuse, arXiv 2609.13612).

Layout of the package:

* ``csrc/``     -- HIP kernels for gfx950 and the C-ABI host code that
                   launches them (built into ``lib/libattnfuse.so``);
* ``_lib``      -- ctypes loader for that library (fails loudly if missing);
* ``api``       -- thin Python binding with the C-ABI's names: argument
                   marshalling only, every step runs in the HIP kernels;
* ``inputs``    -- seeded synthetic input generators (no method arithmetic);
* ``workloads`` -- the named workload shapes and their FLOP / byte counts;
* ``build``     -- the hipcc build of the library.

Importing the package loads nothing native; ``api`` loads the library on
first use.
"""
__version__ = "0.1.0"
