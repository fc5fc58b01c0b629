"""ctypes view of libbsa.so (the C ABI declared in include/bsa.h).

Loading fails loudly when the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbsa.so")

BSA_OK, BSA_ERR_INVALID_ARGUMENT, BSA_ERR_UNSUPPORTED, BSA_ERR_WORKSPACE_TOO_SMALL, BSA_ERR_HIP = range(5)
BSA_F32, BSA_BF16 = 0, 1
BSA_POOL_MLP, BSA_POOL_MEAN = 0, 1
BSA_QC_MEAN, BSA_QC_MLP = 0, 1


class bsa_params_t(C.Structure):
    _fields_ = [
        ("batch", C.c_int32), ("n", C.c_int32), ("heads", C.c_int32), ("head_dim", C.c_int32),
        ("ball_size", C.c_int32), ("cmp_block", C.c_int32), ("cmp_stride", C.c_int32),
        ("slc_block", C.c_int32), ("topk", C.c_int32), ("group_size", C.c_int32),
        ("mask_own_ball", C.c_int32), ("store_lse", C.c_int32), ("deterministic", C.c_int32),
        ("kv_pool", C.c_int32), ("dtype", C.c_int32), ("softmax_scale", C.c_float),
        ("q_coarsen", C.c_int32), ("group_compression", C.c_int32),
    ]


class bsa_mlp_t(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("b1", C.c_void_p), ("w2", C.c_void_p), ("b2", C.c_void_p)]


bsa_mlp_grad_t = bsa_mlp_t


class bsa_saved_t(C.Structure):
    _fields_ = [
        ("sel_idx", C.c_void_p), ("lse", C.c_void_p), ("o_branch", C.c_void_p),
        ("kcmp", C.c_void_p), ("vcmp", C.c_void_p), ("hid_k", C.c_void_p), ("hid_v", C.c_void_p),
        ("cvalid", C.c_void_p), ("qcmp", C.c_void_p), ("hid_q", C.c_void_p), ("ocmp", C.c_void_p),
        ("o_cmp", C.c_void_p),
    ]


_BLOCK_W = ("g1", "wqkv", "wg", "wo", "g2", "w1", "w3", "w2")


class bsa_block_weights_t(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _BLOCK_W] + [("phi_k", bsa_mlp_t), ("phi_v", bsa_mlp_t), ("phi_q", bsa_mlp_t)]


bsa_block_grads_t = bsa_block_weights_t


class bsa_block_saved_t(C.Structure):
    _fields_ = [("layer", bsa_saved_t)] + [(n, C.c_void_p) for n in (
        "rstd1", "rstd2", "xn1", "gate", "q", "k", "v", "o", "h", "xn2", "uw", "a")]


_SIGS = {
    "bsa_status_string": (C.c_char_p, [C.c_int]),
    "bsa_last_error": (C.c_char_p, []),
    "bsa_timing_enable": (C.c_int, [C.c_int32]),
    "bsa_timing_select": (C.c_int, [C.c_char_p]),
    "bsa_set_streams": (C.c_int, [C.c_int32]),
    "bsa_timing_query": (C.c_int, [C.c_char_p, C.POINTER(C.c_double), C.POINTER(C.c_int32)]),
    "bsa_ball_tree_workspace_bytes": (C.c_size_t, [C.c_int64, C.c_int64, C.c_int32, C.c_int32]),
    "bsa_build_ball_tree": (C.c_int, [C.c_void_p, C.c_int64, C.c_int32, C.c_int64, C.c_int32, C.c_void_p,
                                      C.c_void_p, C.c_size_t, C.c_void_p]),
    "bsa_build_ball_tree_noalloc": (C.c_int, [C.c_void_p, C.c_int64, C.c_int32, C.c_int64, C.c_int32, C.c_void_p,
                                              C.c_void_p]),
    "bsa_permute": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, C.c_int64, C.c_int32, C.c_int32, C.c_int32,
                              C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]),
    "bsa_unpermute": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, C.c_int64, C.c_int32, C.c_int32, C.c_int32,
                                C.c_int32, C.c_void_p, C.c_void_p]),
    "bsa_sizes": (C.c_int, [C.POINTER(bsa_params_t), C.POINTER(C.c_size_t), C.POINTER(C.c_size_t),
                            C.POINTER(C.c_size_t)]),
    "bsa_saved_view": (C.c_int, [C.POINTER(bsa_params_t), C.c_void_p, C.POINTER(bsa_saved_t)]),
    "bsa_forward": (C.c_int, [C.POINTER(bsa_params_t), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                              C.POINTER(bsa_mlp_t), C.POINTER(bsa_mlp_t), C.POINTER(bsa_mlp_t), C.c_void_p,
                              C.POINTER(bsa_saved_t), C.c_void_p, C.c_size_t, C.c_void_p]),
    "bsa_backward": (C.c_int, [C.POINTER(bsa_params_t), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                               C.POINTER(bsa_mlp_t), C.POINTER(bsa_mlp_t), C.POINTER(bsa_mlp_t),
                               C.POINTER(bsa_saved_t), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                               C.POINTER(bsa_mlp_grad_t), C.POINTER(bsa_mlp_grad_t), C.POINTER(bsa_mlp_grad_t),
                               C.c_void_p, C.c_size_t, C.c_void_p]),
    "bsa_block_sizes": (C.c_int, [C.POINTER(bsa_params_t), C.c_int32, C.POINTER(C.c_size_t),
                                  C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "bsa_block_saved_view": (C.c_int, [C.POINTER(bsa_params_t), C.c_int32, C.c_void_p,
                                       C.POINTER(bsa_block_saved_t)]),
    "bsa_block_forward": (C.c_int, [C.POINTER(bsa_params_t), C.c_int32, C.POINTER(bsa_block_weights_t), C.c_void_p,
                                    C.c_void_p, C.c_void_p, C.POINTER(bsa_block_saved_t), C.c_void_p, C.c_size_t,
                                    C.c_void_p]),
    "bsa_block_backward": (C.c_int, [C.POINTER(bsa_params_t), C.c_int32, C.POINTER(bsa_block_weights_t),
                                     C.c_void_p, C.c_void_p, C.POINTER(bsa_block_saved_t), C.c_void_p, C.c_void_p,
                                     C.POINTER(bsa_block_grads_t), C.c_void_p, C.c_size_t, C.c_void_p]),
}

_lib = None


def load() -> C.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2506_12541_amd.build`")
        lib = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


class BsaError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        self.status = status
        msg = lib.bsa_status_string(status).decode()
        detail = lib.bsa_last_error().decode()
        super().__init__(f"{where}: {msg}: {detail}")


def check(status: int, where: str) -> None:
    if status != BSA_OK:
        raise BsaError(status, where)
