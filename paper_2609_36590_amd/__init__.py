"""SEED draft-verify decoding on AMD Instinct MI355X (gfx950).

``synth`` draws the seeded synthetic inputs, ``build`` compiles the HIP library in-tree and
``binding`` is the thin ctypes layer over its C ABI (include/seed.h). Importing the package loads
nothing; ``binding.load_library()`` fails loudly when the library has not been built.
"""
