"""PARD parallel-draft speculative decoding on AMD Instinct MI355X (gfx950).

The compute path is the HIP library ``libpard.so`` (sources in ``csrc/``,
C ABI in ``include/pard.h``); ``binding`` is its ctypes wrapper.  The binding
is imported lazily so that host-only tools (e.g. ``bytes_model``) work before
the library is built.
"""


def load_binding():
    from . import binding
    return binding
