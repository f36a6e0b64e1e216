"""AgentKVShift reuse prefill on AMD MI355X (gfx950).

`akvs` is the ctypes binding of libakvs.so (same names as the C ABI in include/akvs.h);
`runtime.Engine` allocates outputs and workspaces with torch and calls it. Build the
library with `python -m paper_2607_21604_amd.build`.
"""
from . import akvs  # noqa: F401

__all__ = ["akvs"]
