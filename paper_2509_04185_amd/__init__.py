"""MI355X (gfx950) Set Block Decoding decode step: HIP kernels behind a C ABI (libsbd.so).

``Sbd`` wraps one library context; see ``include/sbd.h`` for the semantics of each call.
"""
from .binding import (LIB_PATH, SIGNATURES, ModelConfig, Sbd, SbdError, load_library,
                      make_config, status_string, workspace_bytes)
from .sampler import sample_blocks

__all__ = ["LIB_PATH", "SIGNATURES", "ModelConfig", "Sbd", "SbdError", "load_library",
           "make_config", "sample_blocks", "status_string", "workspace_bytes"]
