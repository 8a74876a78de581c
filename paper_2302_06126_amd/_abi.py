"""ctypes mirror of include/tag.h.

Functions keep the C names; they take plain ints/pointers and the ctypes
structures below.  Nothing here computes anything of the method: every step
runs in libtag.so's HIP kernels.  Loading fails loudly when the library has
not been built.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# TAG_LIBRARY selects another build of the same sources (the CPU sanitizer
# builds of paper_2302_06126_amd/sanitize.py); the default is the in-tree library
LIB_PATH = os.environ.get("TAG_LIBRARY") or os.path.join(_HERE, "libtag.so")

TAG_OK, TAG_EINVAL, TAG_ERANGE, TAG_EDUP, TAG_ESHAPE, TAG_ENOSPACE, TAG_EHIP = 0, -1, -2, -3, -4, -5, -6
TAG_F32, TAG_BF16 = 0, 1
STATUS_NAMES = {0: "TAG_OK", -1: "TAG_EINVAL", -2: "TAG_ERANGE", -3: "TAG_EDUP", -4: "TAG_ESHAPE",
                -5: "TAG_ENOSPACE", -6: "TAG_EHIP"}

EXPORTS = ("tag_graph_plan", "tag_graph_build", "tag_graph_get_info", "tag_graph_export",
           "tag_graph_destroy", "tag_gnn_workspace", "tag_gnn_forward", "tag_gnn_decide_workspace",
           "tag_gnn_decide", "tag_last_error", "tag_version", "tag_profile_begin", "tag_profile_end",
           "tag_gnn_decide_full_workspace", "tag_gnn_decide_full", "tag_gnn_decide_noalloc_max_bytes",
           "tag_gnn_decide_noalloc")
# include/tag_search.h
SEARCH_EXPORTS = ("tag_search_problem_create", "tag_search_problem_destroy", "tag_search_order",
                  "tag_search_evaluate", "tag_mcts_create", "tag_mcts_destroy", "tag_mcts_select",
                  "tag_mcts_update", "tag_mcts_root_stats", "tag_mcts_best_path", "tag_mcts_size",
                  "tag_search_device_bytes", "tag_search_upload", "tag_search_pack", "tag_search_features",
                  "tag_search_run_workspace", "tag_search_run", "tag_simulate", "tag_simulate_batch",
                  "tag_search_set_model", "tag_search_link_features")

# include/tag_train.h
TRAIN_EXPORTS = ("tag_train_workspace", "tag_train_step")

# kernel stages (include/tag_profile.h)
STAGE_NAMES = ("graph_build", "encode", "transform", "agg_op_op", "agg_op_dev", "agg_dev_op", "agg_dev_merge",
               "dev_prep", "decide", "bwd_decoder", "bwd_scores", "bwd_softmax", "bwd_messages", "bwd_dh", "bwd_dw")
FORWARD_STAGES = STAGE_NAMES[:9]
TRAIN_STAGES = STAGE_NAMES[9:]

_P32 = C.POINTER(C.c_int32)
_P64 = C.POINTER(C.c_int64)
_PF = C.c_void_p


class tag_graph_desc(C.Structure):
    _fields_ = [("n_graphs", C.c_int32), ("n_op", _P32), ("n_dev", _P32),
                ("oo_off", _P64), ("dd_off", _P64), ("od_off", _P64),
                ("oo_src", C.c_void_p), ("oo_dst", C.c_void_p),
                ("dd_a", C.c_void_p), ("dd_b", C.c_void_p),
                ("od_op", C.c_void_p), ("od_dev", C.c_void_p)]


class tag_graph_info(C.Structure):
    _fields_ = [("n_graphs", C.c_int32), ("max_dev", C.c_int32), ("n_op", C.c_int64), ("n_dev", C.c_int64),
                ("e_oo", C.c_int64), ("e_dd", C.c_int64), ("e_od", C.c_int64),
                ("rows", C.c_int64 * 4), ("nnz", C.c_int64 * 4), ("max_degree", C.c_int32 * 4)]


class tag_model_dims(C.Structure):
    _fields_ = [("f", C.c_int32), ("heads", C.c_int32), ("layers", C.c_int32), ("f_op", C.c_int32),
                ("f_dev", C.c_int32), ("dec_hidden", C.c_int32), ("dtype", C.c_int32),
                ("gamma_same", C.c_float), ("gamma_cross", C.c_float), ("leaky_slope", C.c_float),
                ("sigma", C.c_int32), ("relations", C.c_int32), ("edge_act", C.c_int32),
                ("head_mode", C.c_int32)]


class tag_weights(C.Structure):
    _fields_ = [("enc_op_w", _PF), ("enc_op_b", _PF), ("enc_dev_w", _PF), ("enc_dev_b", _PF),
                ("enc_edge_w", _PF * 3), ("enc_edge_b", _PF * 3),
                ("layer_w", _PF), ("layer_b", _PF), ("att_src", _PF), ("att_dst", _PF),
                ("dec_w1", _PF), ("dec_b1", _PF), ("dec_w2", _PF), ("dec_b2", _PF)]


class tag_features(C.Structure):
    _fields_ = [("n_replicas", C.c_int32), ("x_op", _PF), ("x_dev", _PF), ("x_oo", _PF), ("x_dd", _PF),
                ("x_od", _PF), ("stride_oo", C.c_int64), ("stride_dd", C.c_int64), ("stride_od", C.c_int64)]


class tag_slices(C.Structure):
    _fields_ = [("n_slices", C.c_int32), ("mask", C.c_void_p), ("option", C.c_void_p)]


class tag_grads(C.Structure):
    _fields_ = tag_weights._fields_


class tag_train_batch(C.Structure):
    _fields_ = [("n_query", C.c_int32), ("query_rep", _PF), ("query_graph", _PF), ("query_op", _PF),
                ("target", _PF)]


class tag_search_problem_desc(C.Structure):
    _fields_ = [("n_op", C.c_int32), ("n_dev", C.c_int32), ("n_groups", C.c_int32), ("n_slices", C.c_int32),
                ("f_op", C.c_int32), ("group_of", C.c_void_p), ("op_type", C.c_void_p),
                ("op_flops", C.c_void_p), ("op_bytes", C.c_void_p), ("op_params", C.c_void_p),
                ("dev_tflops", C.c_void_p), ("dev_mem_gb", C.c_void_p), ("dev_intra_gbs", C.c_void_p),
                ("e_dd", C.c_int64), ("dd_a", C.c_void_p), ("dd_b", C.c_void_p), ("dd_gbs", C.c_void_p),
                ("e_oo", C.c_int64), ("oo_src", C.c_void_p), ("oo_dst", C.c_void_p),
                ("e_od", C.c_int64), ("od_op", C.c_void_p), ("od_dev", C.c_void_p),
                ("slice_mask", C.c_void_p), ("slice_option", C.c_void_p)]


class tag_search_run_args(C.Structure):
    _fields_ = [("problem", C.c_void_p), ("tree", C.c_void_p), ("graph", C.c_void_p), ("dims", C.c_void_p),
                ("weights", C.c_void_p), ("x_oo", C.c_void_p), ("x_dd", C.c_void_p), ("slices", C.c_void_p),
                ("batch", C.c_int32), ("rounds", C.c_int32), ("pipelined", C.c_int32),
                ("workspace", C.c_void_p), ("ws_bytes", C.c_size_t), ("host_buf", C.c_void_p),
                ("host_bytes", C.c_size_t), ("depth_out", C.c_void_p), ("path_out", C.c_void_p),
                ("reward_out", C.c_void_p), ("prior_out", C.c_void_p)]


class tag_sim_out(C.Structure):
    _fields_ = [("iter_time", C.c_double), ("valid", C.c_int32), ("oom", C.c_int32), ("n_tasks", C.c_int64),
                ("group_makespan", _PF), ("group_idle", _PF), ("dev_peak", _PF), ("dev_idle", _PF),
                ("link_idle", _PF)]


class tag_decision(C.Structure):
    _fields_ = [("mask", C.c_uint64), ("option", C.c_int32), ("replicas", C.c_int32),
                ("sync", C.c_int32), ("sfb", C.c_int32)]


_lib = None


def load() -> C.CDLL:
    """Load libtag.so (built in-tree by paper_2302_06126_amd/build.py)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2302_06126_amd.build` "
                           "(the HIP library is required; there is no fallback)")
    lib = C.CDLL(LIB_PATH)
    S = C.c_int32
    vp = C.c_void_p
    szp = C.POINTER(C.c_size_t)
    lib.tag_graph_plan.argtypes = [C.POINTER(tag_graph_desc), szp, szp]
    lib.tag_graph_build.argtypes = [C.POINTER(tag_graph_desc), vp, C.c_size_t, vp, C.c_size_t, vp,
                                    C.POINTER(vp)]
    lib.tag_graph_get_info.argtypes = [vp, C.POINTER(tag_graph_info)]
    lib.tag_graph_export.argtypes = [vp, S, vp, vp, vp]
    lib.tag_graph_destroy.argtypes = [vp]
    lib.tag_graph_destroy.restype = None
    lib.tag_gnn_workspace.argtypes = [vp, C.POINTER(tag_model_dims), S, szp]
    lib.tag_gnn_forward.argtypes = [vp, C.POINTER(tag_model_dims), C.POINTER(tag_weights),
                                    C.POINTER(tag_features), vp, C.c_size_t, vp, vp, vp]
    lib.tag_gnn_decide_workspace.argtypes = [vp, C.POINTER(tag_model_dims), S, S, S, szp]
    lib.tag_gnn_decide.argtypes = [vp, C.POINTER(tag_model_dims), C.POINTER(tag_weights), S, vp, vp,
                                   C.POINTER(tag_slices), S, vp, vp, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]
    for name in ("tag_graph_plan", "tag_graph_build", "tag_graph_get_info", "tag_graph_export",
                 "tag_gnn_workspace", "tag_gnn_forward", "tag_gnn_decide_workspace", "tag_gnn_decide"):
        getattr(lib, name).restype = S
    lib.tag_last_error.restype = C.c_char_p
    lib.tag_last_error.argtypes = []
    lib.tag_version.restype = C.c_char_p
    lib.tag_version.argtypes = []
    lib.tag_profile_begin.argtypes = [S, S]
    lib.tag_profile_begin.restype = S
    lib.tag_profile_end.argtypes = [C.POINTER(C.c_double), C.POINTER(C.c_int32)]
    lib.tag_profile_end.restype = S
    # include/tag_search.h
    lib.tag_search_problem_create.argtypes = [C.POINTER(tag_search_problem_desc), C.POINTER(vp)]
    lib.tag_search_problem_destroy.argtypes = [vp]
    lib.tag_search_problem_destroy.restype = None
    lib.tag_search_order.argtypes = [vp, vp, vp]
    lib.tag_search_evaluate.argtypes = [vp, vp, S, C.POINTER(C.c_double), C.POINTER(C.c_double),
                                        C.POINTER(C.c_int32)]
    lib.tag_mcts_create.argtypes = [S, S, C.c_double, C.c_double, C.POINTER(vp)]
    lib.tag_mcts_destroy.argtypes = [vp]
    lib.tag_mcts_destroy.restype = None
    lib.tag_mcts_select.argtypes = [vp, S, vp, vp, vp]
    lib.tag_mcts_update.argtypes = [vp, S, vp, vp, vp, vp, vp]
    lib.tag_mcts_root_stats.argtypes = [vp, vp, vp]
    lib.tag_mcts_best_path.argtypes = [vp, vp, C.POINTER(C.c_int32)]
    lib.tag_mcts_size.argtypes = [vp, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]
    lib.tag_search_device_bytes.argtypes = [vp, szp, szp]
    lib.tag_search_upload.argtypes = [vp, vp, C.c_size_t, vp]
    lib.tag_search_pack.argtypes = [vp, S, vp, vp, S, vp, vp, vp]
    lib.tag_search_features.argtypes = [vp, S, vp, vp, vp, vp, vp, vp]
    lib.tag_search_run_workspace.argtypes = [vp, vp, C.POINTER(tag_model_dims), S, szp, szp]
    lib.tag_search_run.argtypes = [C.POINTER(tag_search_run_args), vp]
    lib.tag_simulate.argtypes = [vp, vp, S, C.POINTER(tag_sim_out)]
    lib.tag_search_set_model.argtypes = [vp, S]
    lib.tag_search_link_features.argtypes = [vp, S, vp, vp, vp, vp]
    lib.tag_simulate_batch.argtypes = [vp, S, vp, vp, S, S, vp, vp]
    lib.tag_train_workspace.argtypes = [vp, C.POINTER(tag_model_dims), S, S, S, szp]
    lib.tag_train_step.argtypes = [vp, C.POINTER(tag_model_dims), C.POINTER(tag_weights), C.POINTER(tag_features),
                                   C.POINTER(tag_slices), C.POINTER(tag_train_batch), C.POINTER(tag_grads),
                                   C.c_float, vp, vp, C.c_size_t, vp]
    for name in TRAIN_EXPORTS:
        getattr(lib, name).restype = S
    lib.tag_gnn_decide_full_workspace.argtypes = [vp, C.POINTER(tag_model_dims), S, S, szp]
    lib.tag_gnn_decide_full.argtypes = [vp, C.POINTER(tag_model_dims), C.POINTER(tag_weights), S, vp, vp, S, vp,
                                        vp, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]
    lib.tag_gnn_decide_full_workspace.restype = S
    lib.tag_gnn_decide_full.restype = S
    lib.tag_gnn_decide_noalloc_max_bytes.argtypes = []
    lib.tag_gnn_decide_noalloc_max_bytes.restype = C.c_size_t
    lib.tag_gnn_decide_noalloc.argtypes = [vp, C.POINTER(tag_model_dims), C.POINTER(tag_weights), S, vp, vp,
                                           C.POINTER(tag_slices), S, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.tag_gnn_decide_noalloc.restype = S
    for name in SEARCH_EXPORTS:
        if name not in ("tag_search_problem_destroy", "tag_mcts_destroy"):
            getattr(lib, name).restype = S
    _lib = lib
    return lib


class TagError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def check(status: int, where: str) -> None:
    if status != TAG_OK:
        raise TagError(status, where, load().tag_last_error().decode(errors="replace"))
