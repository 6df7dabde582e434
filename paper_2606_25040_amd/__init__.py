"""MI355X-native block-sparse attention with a reusable block mask (Chorus II hot path).

The compute path lives in ``libchorus.so`` (hand-written HIP for gfx950, C ABI
declared in ``include/chorus.h``); :mod:`.ops` marshals torch tensors into that
ABI.  Importing the package does not load the library; the first op call does,
and fails loudly if it has not been built.
"""

from .ops import (  # noqa: F401
    BlockMask,
    VisitMap,
    attn_block_mass,
    block_sparse_attn_fwd,
    block_sparse_attn_fwd_bf16,
    block_sparse_attn_fwd_f16,
    block_sparse_attn_fwd_fp8,
    build_block_mask,
    build_block_mask_noalloc,
    load_library,
    mask_coverage,
    plan_block_mask,
    quantize_fp8_blockwise,
    select_block_mask,
    validate_block_mask,
)
