"""MI355X (gfx950) low-bit substitute layers of SubSpec (Sec. 4.1), and the draft-tree
expansion step that follows every draft pass (Sec. 4.2).

The compute path is the native library ``libsubspec.so`` (hand-written HIP,
C ABI in ``include/subspec.h``); this package only marshals arguments to it.
Importing works without a GPU; calling a device entry point needs the library
built for gfx950 and fails loudly when it is missing.
"""
from ._binding import (  # noqa: F401
    SUBSPEC_PATH_AUTO,
    SUBSPEC_PATH_GEMV,
    SUBSPEC_PATH_MFMA,
    SUBSPEC_PATH_MFMA16,
    SUBSPEC_PATH_MFMA32,
    SubspecError,
    library_path,
    load_library,
    subspec_last_error,
    subspec_qdequant,
    subspec_qlinear,
    subspec_qlinear_path,
    subspec_qlinear_noalloc,
    SUBSPEC_NOALLOC_SCRATCH_BYTES,
    subspec_qlinear_plan,
    subspec_qpack,
    subspec_qpack_bytes,
    subspec_qpack_host,
    subspec_quantize,
    subspec_quantize_hqq,
    subspec_reserve,
    subspec_workspace_info,
    subspec_stack_forward,
    subspec_stack_capture,
    subspec_graph_launch,
    subspec_graph_destroy,
    subspec_tree_expand,
    Prefetcher,
    subspec_tree_attention,
    subspec_tree_attention_plan,
    subspec_tree_attention_workspace_bytes,
    subspec_tree_plan,
    subspec_tree_workspace_bytes,
)
