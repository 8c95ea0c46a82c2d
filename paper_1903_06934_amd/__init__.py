"""MI355X-native fp32 convolution training passes (forward, backward-data,
backward-weight) behind a C ABI (include/miconv.h), with a thin ctypes
binding.  The library is loaded on first use; see ``miconv.lib``."""
from .miconv import (MiconvError, conv_bwd_data, conv_bwd_weight, conv_fwd, conv_tune, lib,
                     output_size, plan_clear, plan_count, plan_get, plan_name, plan_set,
                     plan_workspace_size, pool_bwd, pool_fwd, pool_output_size, workspace_size,
                     PASS_FWD, PASS_BWD_DATA, PASS_BWD_WEIGHT)

__all__ = ["MiconvError", "conv_fwd", "conv_bwd_data", "conv_bwd_weight", "conv_tune", "lib",
           "output_size", "plan_clear", "plan_count", "plan_get", "plan_name", "plan_set",
           "plan_workspace_size", "pool_bwd", "pool_fwd", "pool_output_size", "workspace_size",
           "PASS_FWD", "PASS_BWD_DATA", "PASS_BWD_WEIGHT"]
