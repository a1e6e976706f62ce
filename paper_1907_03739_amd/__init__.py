"""MI355X (gfx950) Point-Voxel Convolution forward.

The computation lives in libpvconv.so (HIP kernels behind the C ABI declared in
include/pvconv.h); `binding` marshals torch tensors into those calls and
`network` chains them into the PVCNN segmentation networks.

The binding is imported on first use of one of its names, so that the build
module stays importable before libpvconv.so exists. Using any entry point
without the library raises ImportError: there is no fallback.
"""
import importlib

_BINDING_NAMES = (
    "BF16", "F32", "DeviceLayer", "PVConvError", "pvconv_conv3d", "pvconv_devoxelize",
    "pvconv_forward", "pvconv_forward_workspace_size", "pvconv_maxpool", "pvconv_point_mlp",
    "pvconv_voxelize",
)

__all__ = list(_BINDING_NAMES) + ["DeviceNetwork"]


def __getattr__(name):
    if name in _BINDING_NAMES:
        return getattr(importlib.import_module(".binding", __name__), name)
    if name == "DeviceNetwork":
        return importlib.import_module(".network", __name__).DeviceNetwork
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")
