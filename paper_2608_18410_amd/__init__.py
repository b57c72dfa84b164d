"""librolesub: RoleSub's inference hot path (rotate, route, pack, attend) on MI355X.

The compute runs in hand-written HIP kernels for gfx950 behind a C ABI
(include/rolesub.h); this package is its ctypes binding.
"""
from .rolesub import (  # noqa: F401
    ACT, ADDITIVE, BF16, EXPORTS, F32, LANG, LIB_PATH, MLP2, PROP, THRESHOLD, TOPK, VIS, Budget, Dims,
    Router, RouterDesc, RolesubError, attend, attend_causal, load, make_budget, pack_kv, rotate_values, route,
    rotate_pack, route_workspace_size, status_name, retain_tokens, gather_tokens, allocate_groups,
    route_allocate, route_allocate_workspace_size, full_workspace_size, full_transpose, full_rotate_pack,
    full_values, attend_values, route_noalloc, ROUTE_NOALLOC_MAX_BYTES,
)
