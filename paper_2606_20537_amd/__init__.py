"""Execution-state capsules and the chunked gated linear-attention and gated
delta-rule prefill scans for AMD Instinct MI355X (gfx950).

The product is libcapsule.so (C ABI, include/capsule.h; HIP kernels under
csrc/).  This package holds its build script and a ctypes binding whose
functions carry the C entry points' names.
"""
from ._native import (  # noqa: F401
    CAP_DTYPE_BF16, CAP_DTYPE_F32, CAP_E_ALIGN, CAP_E_DIGEST, CAP_E_HIP, CAP_E_INVAL, CAP_E_NOMEM, CAP_E_SIZE,
    CAP_E_STATE, CAP_E_UNSUPPORTED, CAP_KIND_FIXED, CAP_KIND_POSITIONAL, CAP_MAX_BUFFERS, CAP_MAX_FORK,
    CAP_MAX_GALLERY, CAP_MAX_STAGES, CAP_OK, CAP_TIER_DEVICE, CAP_TIER_HOST, SIGNATURES, CapSet, Capsule, CapsuleError, cap_align_boundary, cap_set_append, cap_set_bind_stage, cap_set_create,
    cap_set_destroy, cap_set_get_position, cap_set_set_position, cap_stage_acquire, cap_stage_invalidate,
    cap_stage_valid_end, cap_status_string, capsule_bytes, capsule_stage_end,
    capsule_digest_tokens, capsule_fork, capsule_gather_restore, capsule_info, capsule_layout_bytes,
    capsule_move, capsule_release, capsule_restore, capsule_snapshot, capsule_tier, gdn_chunked_prefill,
    gdn_chunked_prefill_noalloc, GDN_NOALLOC_SCRATCH_BYTES,
    gdn_decode_step, gdn_workspace_bytes, kv_fp8_dequantize, kv_fp8_quantize, linattn_chunked_prefill,
    linattn_decode_step, load,
)
