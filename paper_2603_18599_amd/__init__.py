"""MI355X (gfx950) speculative-Jacobi step library for SJD-PAC.

The compute path lives in libsjd.so (hand-written HIP); this package only
marshals arguments to its C ABI (include/sjd.h). Importing it does not need a
GPU, but every call that reaches the library needs the built libsjd.so and
fails loudly without it.
"""
from .sjd import (SJD_AC, SJD_PD, SjdError, lib_path, load_library, sjd_status_str,  # noqa: F401
                  sjd_verify, Engine)
