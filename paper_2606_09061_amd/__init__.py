"""MI355X-native mixed prefill/decode paged attention for chunked-prefill serving.

The HIP library (libcpattn.so, built from csrc/ for gfx950) holds the whole
path: the varlen planner, the paged KV append, the bf16-MFMA prefill-chunk
kernel, the split-K decode kernel and the merge pass.  ``binding`` is the
ctypes layer over its C ABI (include/cp_attn.h), re-exported here; the
scheduler (``sched``, ``lprs``, ``serve``) and the decoder layer around the
step (``model``) sit on top of it.
"""

from .binding import (  # noqa: F401
    AttnPlan,
    CpError,
    Desc,
    attn_mixed,
    attn_prepare,
    attn_run,
    check_batch,
    check_block_tables,
    desc_for,
    kv_append,
    make_desc,
    plan_items,
    plan_records,
    plan_summary,
    step_mixed,
    version,
    workspace_bytes,
)
