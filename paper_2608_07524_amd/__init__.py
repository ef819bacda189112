"""DCP hot path on MI355X: packed varlen attention (HIP/CDNA4), per-length
cost profiling and the DCP planner, all behind the C ABI of libdcp.

The Python layer only marshals arguments; see ``_native`` and include/dcp.h.
"""

from ._native import (DCP_ERR_HIP, DCP_ERR_INFEASIBLE, DCP_ERR_INVALID, DCP_ERR_TABLE, DCP_ERR_UNSUPPORTED,
                      DCP_ERR_WORKSPACE, DCP_OK, PLAN_FLAG_MIN_TIME, PLAN_FLAG_NO_HEAD_FILTER, PLAN_INTER,
                      PLAN_INTRA, CostRow, DCPError, Layer, Plan, PreparedAttention, bwd_workspace_size,
                      default_plan_opts, device_info, fwd_workspace_size, last_error, layer_param_shapes, load, plan,
                      profile_cost, set_kernel_events, simulate, varlen_attn_bwd, varlen_attn_fwd,
                      varlen_attn_fwd_noalloc, work_list)

__all__ = [n for n in dir() if not n.startswith("_")]
