"""MI355X-native hot path of DraftExpert's self-speculative MoE decoding.

The compute lives in ``libdraftexpert.so`` (hand-written HIP for gfx950,
C ABI in ``include/draftexpert.h``).  This package only marshals arguments:
``_lib`` binds every C entry point under its own name; ``model`` composes the
calls into layers and the draft/verify step of a stacked model.
"""
from ._lib import *  # noqa: F401,F403
from ._lib import C_FUNCS, LIB, LIB_PATH, DEError  # noqa: F401
