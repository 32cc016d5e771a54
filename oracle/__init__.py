"""CPU oracle of the DFX calibration hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, exact reference of what FxP-QNet (Shawahna et al., IEEE Access
2022) computes on its hot path: DFX quantization (Eq. 10-13), the
data-structure error (Eq. 14), the exhaustive fractional-length search, the
integer C-Block (conv/FC + bias + Scale + ReLU, Sec. "Integer-Only Inference"
and the text under Fig. "FxP-QNet hardware") and the FxP-QLayer requantization.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU library
``paper_2203_12091_amd``.
"""
from .core import *  # noqa: F401,F403
from . import nets  # noqa: F401
