"""MI355X-native channelwise Clebsch-Gordan tensor product and message-passing
convolution (forward and backward), after "E3J: An Efficient and Open-Source
Backend for Euclidean Equivariant Operations on GPU and TPU".

The compute lives in the HIP library ``libe3mi.so`` (kernels under ``csrc/``,
C ABI in ``include/e3mi.h``); ``e3mi`` is its Python binding.
"""
from .e3mi import (E3Error, Graph, Linear, Plan, RecordTP, conv_bwd, conv_bwd2, conv_bwd_radial, conv_bwd_y, conv_fwd,
                   conv_fwd_radial, conv_fwd_y,
                   conv_radial_workspace_size, conv_workspace_size, sh, sh_bwd, sh_host, tp_bwd, tp_fwd,
                   tp_workspace_size, workspace)

__all__ = ["E3Error", "Graph", "Linear", "Plan", "RecordTP", "conv_bwd", "conv_bwd2", "conv_bwd_radial", "conv_bwd_y", "conv_fwd",
           "conv_fwd_radial", "conv_fwd_y",
           "conv_radial_workspace_size", "conv_workspace_size", "sh", "sh_bwd", "sh_host", "tp_bwd",
           "tp_fwd", "tp_workspace_size", "workspace"]
