"""MI355X-native paged grouped-query decode attention (HIP, gfx950).

The C ABI is declared in include/laminar_decode_attn.h and
include/laminar_kv_append.h, include/laminar_repack.h and
include/laminar_linear.h; ``_native`` binds it
with ctypes under the same names and ``api.PagedDecodeAttention`` owns a plan
and its device workspace. Every step of the computation runs in the HIP
library; there is no CPU fallback.
"""
from . import _native
from ._native import (LaminarAttnDesc, LaminarError, laminar_decode_attn,
                      laminar_decode_attn_merge, laminar_decode_attn_partial,
                      laminar_hbm_copy, laminar_hbm_read,
                      laminar_hbm_read_sink_floats, laminar_kv_append,
                      laminar_plan_bind_workspace,
                      laminar_plan_cascade_members_copy,
                      laminar_plan_cascade_units_copy,
                      laminar_plan_create, laminar_plan_create_cascade,
                      laminar_plan_destroy,
                      laminar_plan_items_copy, laminar_plan_merges_copy,
                      laminar_plan_num_items, laminar_plan_num_merges,
                      laminar_plan_pages_per_item, laminar_plan_waves_per_item,
                      laminar_plan_workspace_bytes, laminar_status_string)
from ._native import (LaminarModelShape, LaminarRolloutState,
                      laminar_migrate_pages, laminar_migration_pairs,
                      laminar_repack_plan, laminar_roofline_batch_bound,
                      laminar_roofline_step_seconds)
from ._native import (laminar_linear, laminar_linear_bf16,
                      laminar_linear_bf16_ex, laminar_linear_bf16_rmsnorm,
                      laminar_linear_pack,
                      laminar_linear_splits, laminar_linear_workspace_bytes)
from .api import (PagedDecodeAttention, SkinnyLinear, kv_append, migrate,
                  rmsnorm, silu_mul)
