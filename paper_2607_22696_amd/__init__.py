"""3D Deformable Slide Attention (MegaSlide-DiT, Section 5.2, Eq. (1)) for MI355X (gfx950).

The operator runs in the hand-written HIP kernels of ``libdsa3d.so`` behind the C ABI
declared in ``include/dsa3d.h``.  This package holds the kernels (``csrc/``), the build
script and a thin binding; PyTorch is used only for device memory and streams.
"""
from ._binding import (  # noqa: F401
    DSA3D_BACKWARD_PHASES, DSA3D_BF16, DSA3D_WIN_BACKWARD_PHASES, DSA3D_F32, DSA3D_MAX_POINTS, DSA3D_OK, EXPORTED, Dsa3dError,
    dsa3d_abi_version, dsa3d_backward, dsa3d_backward_noalloc, dsa3d_backward_timed, dsa3d_backward_workspace_size,
    dsa3d_desc, dsa3d_dwconv3d_backward, dsa3d_dwconv3d_backward_workspace_size,
    dsa3d_dwconv3d_forward, dsa3d_dwconv_desc, dsa3d_forward, dsa3d_pw_backward,
    dsa3d_pw_backward_workspace_size, dsa3d_pw_forward, dsa3d_win_backward,
    dsa3d_win_backward_workspace_size, dsa3d_win_desc, dsa3d_win_forward, load, make_conv_desc,
    make_desc, make_win_desc, status_string)
from .ops import (backward, dwconv3d_backward, dwconv3d_forward, forward, pw_backward,  # noqa: F401
                  pw_forward, win_backward, win_forward)
