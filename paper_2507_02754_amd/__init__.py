"""MI355X (gfx950) causal sliding-window 2-simplicial attention.

The compute lives in libsimplicial_attn.so (hand-written HIP, C ABI in
include/simplicial_attn.h); this package is its thin Python binding plus the
seeded synthetic workloads used by the tests and the benchmark, and a
torch.autograd wrapper (`simplicial_attention`) over the forward and backward
entry points, and the surrounding layer (`SimplicialAttention`: the K, K', V,
V' projections of Section 4 around the kernels) with a small stack that
interleaves it with dot-product attention (`InterleavedStack`).
"""

from .autograd import SimplicialAttnFunction, simplicial_attention  # noqa: F401
from .layer import InterleavedStack, SimplicialAttention  # noqa: F401
from .binding import (  # noqa: F401
    DTYPE_BF16,
    DTYPE_F32,
    SimplicialAttnError,
    load_library,
    simplicial_attn_abi_version,
    simplicial_attn_bwd,
    simplicial_attn_bwd_gqa,
    simplicial_attn_bwd_gqa_workspace_size,
    simplicial_attn_bwd_biased,
    simplicial_attn_bwd_noalloc,
    simplicial_attn_det_bwd,
    simplicial_attn_det_bwd_workspace_size,
    simplicial_attn_det_fwd,
    simplicial_attn_bwd_fused,
    simplicial_attn_bwd_fused_reduce,
    simplicial_attn_bwd_fused_workspace_size,
    simplicial_attn_bwd_key_side,
    simplicial_attn_bwd_preprocess,
    simplicial_attn_bwd_query_side,
    simplicial_attn_bwd_workspace_size,
    simplicial_attn_error_string,
    simplicial_attn_fwd,
    simplicial_attn_fwd_biased,
    simplicial_attn_fwd_gqa,
    simplicial_attn_path_name,
)
