"""MI355X (gfx950) implementation of GraceKV's one-shot KV-cache compression:
segment -> build trees -> score -> select -> pack, as HIP kernels behind a C
ABI (include/gracekv.h).  ``gracekv`` is the ctypes binding."""
from . import gracekv  # noqa: F401
