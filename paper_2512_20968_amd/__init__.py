"""MI355X-native tile compute of Mesh-Attention (arXiv 2512.20968).

Python binding of ``libmesh_attn.so`` (C ABI in ``include/mesh_attn.h``).
The functions carry the C names and do argument marshalling only: shapes and
dtypes of torch tensors are checked against the problem on the host, then the
C entry point runs every step on the GPU.  There is no fallback: if the HIP
library is missing or a call fails, an exception is raised.
"""

from ._binding import (  # noqa: F401
    MA_BF16,
    MA_FP32,
    MA_CLS_EMPTY,
    MA_CLS_PARTIAL,
    MA_CLS_FULL,
    MeshAttnError,
    Problem,
    Run,
    library_path,
    load_library,
    exported_symbols,
    mesh_attn_block_shape,
    mesh_attn_classify,
    mesh_attn_worklist,
    mesh_attn_worklist_kv_major,
    mesh_attn_fwd_workspace_size,
    mesh_attn_bwd_workspace_size,
    mesh_attn_tile_fwd,
    mesh_attn_tile_fwd_noalloc,
    mesh_attn_lse_merge,
    mesh_attn_tile_bwd,
    mesh_attn_chunk_fwd_workspace_size,
    mesh_attn_chunk_fwd,
    mesh_attn_chunk_bwd_workspace_size,
    mesh_attn_chunk_bwd,
    mesh_attn_goo_plan,
    mesh_attn_last_error,
    Chunk,
    GooStep,
    MA_GOO_NONE,
    MA_GOO_AG_Q,
    MA_GOO_AG_KV,
    MA_GOO_RS_Q,
)
