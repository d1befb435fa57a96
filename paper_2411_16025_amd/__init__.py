"""MI355X-native GCN aggregation (SuperGCN, arXiv 2411.16025, Sections 4 and 6).

The work runs in libgcnagg.so (hand-written HIP for gfx950, C ABI declared in
include/gcnagg.h); ``gcnagg`` is its argument-marshalling binding over torch
device tensors.
"""

from .gcnagg import (  # noqa: F401
    EXPORTS, GCN_ADD_SELF_LOOPS, GCN_DT_BF16, GCN_DT_F32, GCN_GEMM_NN, GCN_GEMM_NT, GCN_GEMM_TN,
    GCN_LAYERNORM, GCN_Q8_USE_CSC, GCN_Q_CODES_2BIT, GCN_SYMMETRIZE, GcnError, Graph, LIB_PATH, gcn_aggregate_bwd,
    gcn_aggregate_fwd, gcn_aggregate_fwd_noalloc, gcn_aggregate_fwd_q8halo, gcn_build_csr, gcn_gcn2_step, gcn_gemm_f32,
    gcn_add_rows, gcn_add_rows_q, gcn_graph_bins, gcn_graph_export, gcn_graph_info, gcn_layernorm_quantize,
    gcn_layernorm_bwd, gcn_layernorm_fwd, gcn_normalize, gcn_normalize_mean, gcn_normalize_rc,
    gcn_prepost_split, gcn_profile_enable, gcn_sage3_forward, gcn_sage3_step,
    gcn_profile_read, gcn_quantize_rows_u8, gcn_relu, gcn_relu_bwd, gcn_softmax_xent, lib)
