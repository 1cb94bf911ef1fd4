"""MI355X-native hot path of DraftExpert's self-speculative MoE decoding.

The compute lives in ``libdraftexpert.so`` (hand-written HIP for gfx950,
C ABI in ``include/draftexpert.h``).  This package only marshals arguments:
``_lib`` binds every C entry point under its own name; ``model`` holds a stacked model's
weights for the step calls (``de_spec_step`` and friends).
"""
from ._lib import *  # noqa: F401,F403
from ._lib import C_FUNCS, LIB, LIB_PATH, DEError  # noqa: F401
from .model import DeviceModel  # noqa: F401
