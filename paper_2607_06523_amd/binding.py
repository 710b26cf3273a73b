"""ctypes binding of libdwkv.so: argument marshalling only.

Every computation runs in the library's HIP kernels; torch supplies device
memory and the current stream.  Loading fails loudly when the library is
missing -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libdwkv.so")

MAX_LEVELS = 8
MAX_PROBE_HEADS = 64
F16, BF16 = 0, 1
COEF_F16, COEF_I8 = 0, 1

STATUS = {0: "ok", 1: "null pointer", 2: "inconsistent dimensions", 3: "unsupported shape",
          4: "workspace too small", 5: "malformed cache layout", 6: "HIP runtime error",
          7: "device pointer not 16-byte aligned", 8: "needs more than the static scratch"}


class DwkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS.get(status, status)} (status {status})")
        self.status = status


class Dims(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_layers", C.c_int32), ("window", C.c_int32),
                ("n_kv_heads", C.c_int32), ("n_q_heads", C.c_int32), ("head_dim", C.c_int32),
                ("basis_rank", C.c_int32), ("n_levels", C.c_int32),
                ("levels", C.c_int32 * MAX_LEVELS),
                ("cu_seqlens_host", C.POINTER(C.c_int32)), ("cu_seqlens", C.c_void_p),
                ("total_tokens", C.c_int64), ("res_stride", C.c_int64),
                ("split_tokens", C.c_int32), ("coef_format", C.c_int32)]


class Cache(C.Structure):
    _fields_ = [("basis", C.c_void_p), ("coef_k", C.c_void_p), ("coef_v", C.c_void_p),
                ("rank_code", C.c_void_p),
                ("res_off", C.c_void_p), ("res_idx", C.c_void_p), ("res_val", C.c_void_p),
                ("res_scale", C.c_void_p), ("coef_k_scale", C.c_void_p), ("coef_v_scale", C.c_void_p)]


class Controller(C.Structure):
    _fields_ = [("tol", C.c_float), ("step_down", C.c_float), ("step_up", C.c_float), ("patience", C.c_int32),
                ("theta_min", C.c_float), ("theta_max", C.c_float)]


class Probe(C.Structure):
    _fields_ = [("n_heads", C.c_int32), ("kv_heads_host", C.POINTER(C.c_int32)),
                ("k_ref", C.c_void_p), ("v_ref", C.c_void_p), ("eps", C.c_float),
                ("err", C.c_void_p), ("out_ref", C.c_void_p), ("n_pos", C.c_int32), ("q_prev", C.c_void_p)]


EXPORTS = ["dwkv_abi_version", "dwkv_status_str", "dwkv_split_tokens", "dwkv_decode_kernel", "dwkv_workspace_bytes",
           "dwkv_decode_launches", "dwkv_decode", "dwkv_decode_partials", "dwkv_decode_merge",
           "dwkv_static_scratch_bytes", "dwkv_decode_noalloc", "dwkv_route_workspace_bytes", "dwkv_route",
           "dwkv_route_range", "dwkv_route_budget_workspace_bytes", "dwkv_route_budget", "dwkv_compress", "dwkv_features_workspace_bytes", "dwkv_decode_features", "dwkv_probe_feature", "dwkv_probe_schedule",
           "dwkv_decode_append_workspace_bytes", "dwkv_decode_append_launches", "dwkv_decode_append",
           "dwkv_controller_update", "dwkv_sketch_workspace_bytes", "dwkv_sketch_basis", "dwkv_materialize", "dwkv_dense_workspace_bytes",
           "dwkv_dense_decode", "dwkv_residual_map",
           "dwkv_validate_workspace_bytes", "dwkv_validate", "dwkv_hbm_read_blocks", "dwkv_hbm_read"]

_lib = None


ABI_VERSION = 4      # DWKV_ABI_VERSION of the structures above


def load(path: str = LIB_PATH):
    """Load libdwkv.so (raises when it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with paper_2607_06523_amd.build.build()")
    lib = C.CDLL(path)
    P = C.POINTER
    lib.dwkv_abi_version.restype = C.c_int32
    if lib.dwkv_abi_version() != ABI_VERSION:
        raise ImportError(f"{path} has ABI version {lib.dwkv_abi_version()}, the binding expects "
                          f"{ABI_VERSION}: rebuild it with paper_2607_06523_amd.build.build()")
    lib.dwkv_status_str.restype = C.c_char_p
    lib.dwkv_status_str.argtypes = [C.c_int]
    lib.dwkv_split_tokens.restype = C.c_int32
    lib.dwkv_split_tokens.argtypes = [P(Dims)]
    lib.dwkv_decode_kernel.restype = C.c_int32
    lib.dwkv_decode_kernel.argtypes = [P(Dims)]
    lib.dwkv_workspace_bytes.restype = C.c_size_t
    lib.dwkv_workspace_bytes.argtypes = [P(Dims), P(Probe)]
    lib.dwkv_decode_launches.restype = C.c_int32
    lib.dwkv_decode_launches.argtypes = [P(Dims), P(Probe)]
    lib.dwkv_decode.restype = C.c_int
    lib.dwkv_decode.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_int32, C.c_float,
                                C.c_void_p, P(Probe), C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_decode_partials.restype = C.c_int
    lib.dwkv_decode_partials.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_int32, C.c_float,
                                         P(Probe), C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_decode_merge.restype = C.c_int
    lib.dwkv_decode_merge.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, P(Probe), C.c_void_p,
                                      C.c_size_t, C.c_void_p]
    lib.dwkv_static_scratch_bytes.restype = C.c_size_t
    lib.dwkv_static_scratch_bytes.argtypes = []
    lib.dwkv_decode_noalloc.restype = C.c_int
    lib.dwkv_decode_noalloc.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_int32, C.c_float,
                                        C.c_void_p, P(Probe), C.c_void_p]
    lib.dwkv_route_workspace_bytes.restype = C.c_size_t
    lib.dwkv_route_workspace_bytes.argtypes = [P(Dims)]
    lib.dwkv_route.restype = C.c_int
    lib.dwkv_route.argtypes = [P(Dims), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                               C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_route_range.restype = C.c_int
    lib.dwkv_route_range.argtypes = [P(Dims), C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_int64,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_route_budget_workspace_bytes.restype = C.c_size_t
    lib.dwkv_route_budget_workspace_bytes.argtypes = [P(Dims)]
    lib.dwkv_route_budget.restype = C.c_int
    lib.dwkv_route_budget.argtypes = [P(Dims), C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_int64,
                                      C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_compress.restype = C.c_int
    lib.dwkv_compress.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                  C.c_int64, C.c_int64, C.c_void_p]
    lib.dwkv_features_workspace_bytes.restype = C.c_size_t
    lib.dwkv_features_workspace_bytes.argtypes = [P(Dims)]
    lib.dwkv_decode_features.restype = C.c_int
    lib.dwkv_decode_features.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_int32, C.c_float,
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_decode_append_workspace_bytes.restype = C.c_size_t
    lib.dwkv_decode_append_workspace_bytes.argtypes = [P(Dims)]
    lib.dwkv_decode_append_launches.restype = C.c_int32
    lib.dwkv_decode_append_launches.argtypes = [P(Dims)]
    lib.dwkv_decode_append.restype = C.c_int
    lib.dwkv_decode_append.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_int32, C.c_float, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_probe_schedule.restype = C.c_int32
    lib.dwkv_probe_schedule.argtypes = [C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32, P(C.c_int32),
                                        P(C.c_int32)]
    lib.dwkv_probe_feature.restype = C.c_int
    lib.dwkv_probe_feature.argtypes = [P(Dims), C.c_int32, C.c_int32, P(C.c_int32), C.c_void_p, C.c_int32,
                                       C.c_void_p, C.c_void_p]
    lib.dwkv_controller_update.restype = C.c_int
    lib.dwkv_controller_update.argtypes = [P(Controller), C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                           C.c_void_p]
    lib.dwkv_sketch_workspace_bytes.restype = C.c_size_t
    lib.dwkv_sketch_workspace_bytes.argtypes = [P(Dims), C.c_int64]
    lib.dwkv_sketch_basis.restype = C.c_int
    lib.dwkv_sketch_basis.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_int64,
                                      C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_materialize.restype = C.c_int
    lib.dwkv_materialize.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.dwkv_dense_workspace_bytes.restype = C.c_size_t
    lib.dwkv_dense_workspace_bytes.argtypes = [P(Dims)]
    lib.dwkv_dense_decode.restype = C.c_int
    lib.dwkv_dense_decode.argtypes = [P(Dims), C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_float,
                                      C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.dwkv_residual_map.restype = C.c_int
    lib.dwkv_residual_map.argtypes = [P(Dims), P(Cache), C.c_int32, C.c_int32, C.c_int32, C.c_int64,
                                      C.c_int64, C.c_void_p, C.c_void_p]
    lib.dwkv_hbm_read_blocks.restype = C.c_int32
    lib.dwkv_hbm_read_blocks.argtypes = []
    lib.dwkv_hbm_read.restype = C.c_int
    lib.dwkv_hbm_read.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p, C.c_int32, C.c_void_p]
    lib.dwkv_validate_workspace_bytes.restype = C.c_size_t
    lib.dwkv_validate.restype = C.c_int
    lib.dwkv_validate.argtypes = [P(Dims), P(Cache), P(C.c_int64), C.c_void_p, C.c_size_t, C.c_void_p]
    _lib = lib
    return lib


def check(status: int, where: str):
    if status != 0:
        raise DwkvError(status, where)


def make_dims(*, batch, n_layers, window, n_kv_heads, n_q_heads, head_dim, basis_rank, levels,
              cu_seqlens_host, cu_seqlens_dev_ptr, total_tokens, res_stride, split_tokens=0, coef_format=0):
    """Fill a Dims struct; returns (dims, keepalive) -- keep both alive while in use."""
    cu = np.ascontiguousarray(cu_seqlens_host, dtype=np.int32)
    d = Dims()
    d.batch, d.n_layers, d.window = batch, n_layers, window
    d.n_kv_heads, d.n_q_heads, d.head_dim, d.basis_rank = n_kv_heads, n_q_heads, head_dim, basis_rank
    d.n_levels = len(levels)
    for i, v in enumerate(levels[:MAX_LEVELS]):
        d.levels[i] = int(v)
    d.cu_seqlens_host = cu.ctypes.data_as(C.POINTER(C.c_int32))
    d.cu_seqlens = cu_seqlens_dev_ptr
    d.total_tokens, d.res_stride, d.split_tokens = total_tokens, res_stride, split_tokens
    d.coef_format = coef_format
    return d, cu
