"""MI355X-native fast-feedforward (FFF) inference: conditional matrix multiplication on gfx950.

The compute lives in ``libfff.so`` (HIP kernels behind the C ABI of
``include/fff.h``); this package is its ctypes binding plus the seeded
synthetic-input generators and the named workloads.
"""
from .fff import (  # noqa: F401
    FffArgs, FffBackwardArgs, FffError, FffLayer, backward, backward_workspace_bytes, describe, describe_stack,
    forward, forward_plain, forward_stack, forward_static, from_numpy, load_library, make_args, status_str, to_numpy, version,
    workspace_bytes,
)
