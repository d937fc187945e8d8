"""MI355X (gfx950) SS2D selective scan: full and VMeanba channel-mean variants.

The computation lives in libvmb.so (hand-written HIP kernels behind the C ABI
declared in include/vmb.h); ``paper_2412_16602_amd.vmb`` is its ctypes
binding. Importing this package does not load the library; the first call
does, and fails loudly if it has not been built.
"""
from .vmb import (VMB_BF16, VMB_F32, VMB_LAYOUT_2D, VMB_LAYOUT_SEQ, VmbError,  # noqa: F401
                  abi_version, load_library, vmb_cross_merge, vmb_cross_scan,
                  vmb_mean_scan_fwd, vmb_scan_workspace_bytes, vmb_selective_scan_fwd)
