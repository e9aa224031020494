"""SSM (Structured Suffix Modeling) block-wise denoising step on MI355X.

The compute path lives in libssm.so (HIP, gfx950) behind the C ABI of
include/ssm.h; this package holds the build script, a ctypes binding with the
same call names and the host-side generation loop.
"""
from ._lib import SSMError, lib  # noqa: F401
