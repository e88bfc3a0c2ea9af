"""Wan-Streamer v0.2 performer unit attention on MI355X (gfx950).

The compute lives in ``libws.so`` (HIP kernels behind a C ABI declared in
``include/ws.h``).  ``paper_2607_04443_amd.ws`` is the thin ctypes binding with
the same names; importing it loads the library and fails loudly when it is
missing.  ``paper_2607_04443_amd.synth`` holds the seeded input generators.
"""
