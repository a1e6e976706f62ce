"""MI355X (gfx950) Point-Voxel Convolution forward.

The computation lives in libpvconv.so (HIP kernels behind the C ABI declared in
include/pvconv.h); `binding` marshals torch tensors into those calls and
`network` chains them into the PVCNN segmentation networks.
"""
from .binding import (  # noqa: F401
    BF16, F32, DeviceLayer, PVConvError, pvconv_conv3d, pvconv_devoxelize, pvconv_forward,
    pvconv_forward_workspace_size, pvconv_maxpool, pvconv_point_mlp, pvconv_voxelize,
)
