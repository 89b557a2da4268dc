"""MI355X-native (gfx950) flow-matching action-expert denoise loop.

The HIP library libvla.so (built by paper_2606_08094_amd.build) exposes the C
ABI of include/vla.h; paper_2606_08094_amd.vla is its ctypes binding.
"""
from . import vla  # noqa: F401
