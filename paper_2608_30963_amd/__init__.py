"""kvx: cross-model KV-cache translation on AMD Instinct MI355X (gfx950).

The package is deliberately small:

* ``kvx``    -- Python binding of the C-ABI library ``libkvx.so`` (argument
               marshalling only; every step of the translation runs in HIP
               kernels behind ``kvx_translate``).
* ``synth``  -- seeded synthetic inputs shaped like the paper's model pairs.
* ``build``  -- compiles ``csrc/`` into ``libkvx.so`` with hipcc for gfx950.

Importing the package loads nothing native; ``kvx.load()`` does.
"""

__all__ = ["kvx", "synth", "build"]
