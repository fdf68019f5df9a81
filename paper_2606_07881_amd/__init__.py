"""MI355X (gfx950) implementation of one PACI pipeline stage.

``configs`` and ``inputs`` are pure Python. The stage itself lives in the HIP
library ``libpaci_stage.so`` built from ``csrc/`` and is reached through
``binding`` (ctypes); importing ``binding`` fails loudly when the library is
missing.
"""
