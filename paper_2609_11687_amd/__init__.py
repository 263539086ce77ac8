"""MI355X-native Kashin-DCT decomposition and 2-bit clustering (HIP, gfx950).

The compute path lives in the C-ABI library ``libkashin.so`` (built from
``csrc/``); ``kashin`` is its thin ctypes binding.  ``synth`` draws seeded
synthetic weight matrices.  Importing the package does not load the library;
``kashin.lib()`` does, and raises if it has not been built.
"""
