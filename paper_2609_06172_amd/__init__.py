"""MI355X-native tensor-granular prefetch runtime (C-ABI library + binding).

The library ``libautouvm.so`` holds the planner, the transfer engine and the
HIP kernels; this package only marshals arguments to it.
"""
from .capi import AuvmError, Context, LIB_PATH, SYMBOLS, lib  # noqa: F401
