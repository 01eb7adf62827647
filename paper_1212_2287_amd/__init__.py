"""MI355X (gfx950) tree-ensemble scorer: hand-written HIP kernels behind the C ABI of
``include/tree_ens.h``, with a thin ctypes binding of the same names."""
from ._binding import (  # noqa: F401
    TREE_ENS_E_ARG, TREE_ENS_E_DEVICE, TREE_ENS_E_MODEL, TREE_ENS_E_NOMEM, TREE_ENS_E_SHAPE, TREE_ENS_OK,
    TREE_ENS_RIGHT_IF_GE, TREE_ENS_RIGHT_IF_GT, TREE_ENS_CODEGEN, LIB_PATH, TreeEnsError, TreeEnsLibraryMissing, TreeEnsemble,
    header_functions, load_library, tree_ens_codegen_source, tree_ens_create, tree_ens_create_multi, tree_ens_destroy,
    tree_ens_feature_usage, tree_ens_info, tree_ens_kernel_time, tree_ens_kernel_timing, tree_ens_last_error,
    tree_ens_outputs, tree_ens_predict,
    tree_ens_predict_leaves, tree_ens_predict_noalloc, tree_ens_predict_topk, tree_ens_topk,
)
