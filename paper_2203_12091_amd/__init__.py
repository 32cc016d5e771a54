"""libfxpq: the MI355X (gfx950) DFX calibration hot path of FxP-QNet.

``fxpq`` is the thin ctypes binding of the C ABI in ``include/fxpq.h``;
``nets`` runs whole calibration forwards through it.
"""
from . import fxpq  # noqa: F401
