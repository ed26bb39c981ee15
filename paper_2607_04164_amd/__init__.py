"""MI355X-native grouped ("full-brownout") MoE layer forward.

The work runs in ``libbrownout_moe.so`` (HIP kernels for gfx950) behind the C
ABI in ``include/brownout_moe.h``; this package holds its build step, a thin
ctypes binding and the seeded workload generator used by tests and benchmarks.
"""
from .binding import (BMOE_BF16, BMOE_F32, BmoeError, Desc, LayerForward, combine, dispatch, ffn,
                      ffn_down, ffn_gate_up,
                      load_library, make_desc, new_dispatch_workspace, route, validate,
                      validate_map, workspace_bytes)

__all__ = ["BMOE_BF16", "BMOE_F32", "BmoeError", "Desc", "LayerForward", "combine", "dispatch", "ffn", "ffn_down", "ffn_gate_up",
           "load_library", "make_desc", "new_dispatch_workspace", "route", "validate", "validate_map",
           "workspace_bytes"]
