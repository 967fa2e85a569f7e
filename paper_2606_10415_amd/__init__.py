"""MI355X-native (gfx950) decoder-layer training kernels behind a C ABI.

``paper_2606_10415_amd.lt`` is the ctypes binding of the HIP library
``liblt.so`` (built by ``paper_2606_10415_amd/build.py``); ``synth`` draws the
seeded synthetic inputs.  Importing the package itself loads nothing.
"""
