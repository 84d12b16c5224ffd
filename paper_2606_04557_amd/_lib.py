"""ctypes declarations mirroring include/cas.h."""
from __future__ import annotations

import ctypes
import os

# The in-tree build; CAS_LIB names another build of the same library (the
# host-sanitized one that the host-side tests can run against).
LIB_PATH = os.environ.get("CAS_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcas.so")

CAS_OK = 0
CAS_ERR_INVALID_ARGUMENT = 1
CAS_ERR_UNSUPPORTED = 2
CAS_ERR_ALIGNMENT = 3
CAS_ERR_NOT_PINNED = 4
CAS_ERR_WORKSPACE = 5
CAS_ERR_HIP = 6
CAS_ERR_IO = 7

CAS_DTYPE_BF16 = 0
CAS_DTYPE_FP32 = 1

# Every function include/cas.h declares.
EXPORTS = [
    "cas_prefix_attn_workspace_size", "cas_prefix_attn_fwd", "cas_prefix_attn_bwd",
    "cas_cartridge_stage", "cas_status_string", "cas_last_error_message", "cas_abi_version",
    "cas_set_tuning", "cas_get_tuning", "cas_plan_info", "cas_timing_enable",
    "cas_timing_reset", "cas_timing_read", "cas_adam_lr_scale", "cas_cartridge_adam_workspace_size",
    "cas_cartridge_adam", "cas_paged_decode_workspace_size", "cas_paged_decode_fwd",
    "cas_pool_plan_rotation", "cas_pool_create", "cas_pool_destroy", "cas_pool_host_cartridge",
    "cas_pool_load", "cas_pool_active", "cas_pool_end_step", "cas_pool_flush",
    "cas_prefix_attn_fwd_noalloc", "cas_pool_read_moments",
]


class Segment(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("dk", ctypes.c_void_p),
                ("dv", ctypes.c_void_p), ("len", ctypes.c_int64), ("stride_tok", ctypes.c_int64),
                ("stride_head", ctypes.c_int64)]


class Problem(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("batch", ctypes.c_int32), ("q_len", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("segments", ctypes.POINTER(Segment)), ("seg_offsets", ctypes.POINTER(ctypes.c_int32)),
                ("q_offsets", ctypes.POINTER(ctypes.c_int32))]


class AdamCartridge(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("dk", ctypes.c_void_p),
                ("dv", ctypes.c_void_p), ("m1_k", ctypes.c_void_p), ("m2_k", ctypes.c_void_p),
                ("m1_v", ctypes.c_void_p), ("m2_v", ctypes.c_void_p), ("len", ctypes.c_int64),
                ("stride_tok", ctypes.c_int64), ("stride_head", ctypes.c_int64),
                ("step", ctypes.c_int32), ("frozen_tokens", ctypes.c_int32)]


class AdamConfig(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("warmup_steps", ctypes.c_int32),
                ("warmup_buckets", ctypes.c_int32)]


class DecodeProblem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("softmax_scale", ctypes.c_float), ("page_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("q_offsets", ctypes.POINTER(ctypes.c_int32)),
                ("kv_lens", ctypes.POINTER(ctypes.c_int32)), ("page_offsets", ctypes.POINTER(ctypes.c_int32)),
                ("page_ids", ctypes.POINTER(ctypes.c_int32))]


class PoolConfig(ctypes.Structure):
    _fields_ = [("num_cartridges", ctypes.c_int32), ("lens", ctypes.POINTER(ctypes.c_int64)),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("budget", ctypes.c_int32),
                ("rotate_every", ctypes.c_int32), ("swap_fraction", ctypes.c_float),
                ("frozen_tokens", ctypes.c_int32), ("moment_dir", ctypes.c_char_p)]


class StageCopy(ctypes.Structure):
    _fields_ = [("host_src", ctypes.c_void_p), ("dev_dst", ctypes.c_void_p), ("bytes", ctypes.c_size_t)]


class Tuning(ctypes.Structure):
    _fields_ = [("fwd_splits", ctypes.c_int32), ("dq_splits", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("fwd_splits", ctypes.c_int32), ("dq_splits", ctypes.c_int32),
                ("fwd_workgroups", ctypes.c_int32), ("dkdv_workgroups", ctypes.c_int32),
                ("unique_segments", ctypes.c_int32), ("total_key_tiles", ctypes.c_int32),
                ("max_prefix_len", ctypes.c_int64), ("ws_fwd_bytes", ctypes.c_size_t),
                ("ws_bwd_bytes", ctypes.c_size_t)]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


ABI_VERSION = 4   # CAS_ABI_VERSION of include/cas.h (q_offsets, no-allocation forward, moment file tier)

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libcas.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libcas is not built ({path} missing): run paper_2606_04557_amd.build")
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    P = ctypes.POINTER
    lib.cas_prefix_attn_workspace_size.argtypes = [P(Problem), ctypes.c_int, P(sz)]
    lib.cas_prefix_attn_fwd.argtypes = [P(Problem), vp, vp, vp, vp, vp, vp, sz, vp]
    lib.cas_prefix_attn_bwd.argtypes = [P(Problem), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.cas_prefix_attn_fwd_noalloc.argtypes = [P(Problem), vp, vp, vp, vp, vp, vp]
    lib.cas_cartridge_stage.argtypes = [P(StageCopy), i32, vp, vp]
    lib.cas_status_string.argtypes = [ctypes.c_int]
    lib.cas_status_string.restype = ctypes.c_char_p
    lib.cas_last_error_message.argtypes = []
    lib.cas_last_error_message.restype = ctypes.c_char_p
    lib.cas_abi_version.restype = i32
    if lib.cas_abi_version() != ABI_VERSION:
        raise RuntimeError(f"libcas ABI {lib.cas_abi_version()} at {path}, this binding expects {ABI_VERSION}: rebuild")
    lib.cas_adam_lr_scale.argtypes = [i32, i32, i32]
    lib.cas_adam_lr_scale.restype = ctypes.c_float
    lib.cas_cartridge_adam_workspace_size.argtypes = [P(AdamCartridge), i32, i32, i32, P(sz)]
    lib.cas_cartridge_adam.argtypes = [P(AdamCartridge), i32, i32, i32, P(AdamConfig), vp, sz, vp]
    lib.cas_paged_decode_workspace_size.argtypes = [P(DecodeProblem), P(sz)]
    lib.cas_paged_decode_fwd.argtypes = [P(DecodeProblem), vp, vp, vp, vp, vp, vp, sz, vp]
    u8p = P(ctypes.c_uint8)
    lib.cas_pool_plan_rotation.argtypes = [P(i32), u8p, i32, i32, ctypes.c_float, P(i32), P(i32), P(i32)]
    lib.cas_pool_create.argtypes = [P(PoolConfig), P(vp)]
    lib.cas_pool_destroy.argtypes = [vp]
    lib.cas_pool_host_cartridge.argtypes = [vp, i32, P(AdamCartridge)]
    lib.cas_pool_load.argtypes = [vp, vp]
    lib.cas_pool_active.argtypes = [vp, P(i32), P(AdamCartridge), i32, P(i32)]
    lib.cas_pool_end_step.argtypes = [vp, vp]
    lib.cas_pool_flush.argtypes = [vp, vp]
    lib.cas_pool_read_moments.argtypes = [vp, i32, P(ctypes.c_float)]
    lib.cas_set_tuning.argtypes = [P(Tuning)]
    lib.cas_get_tuning.argtypes = [P(Tuning)]
    lib.cas_plan_info.argtypes = [P(Problem), P(PlanInfo)]
    lib.cas_timing_enable.argtypes = [ctypes.c_int]
    lib.cas_timing_reset.argtypes = []
    lib.cas_timing_read.argtypes = [P(KernelTime), i32, P(i32)]
    for name in ("cas_prefix_attn_workspace_size", "cas_prefix_attn_fwd", "cas_prefix_attn_bwd",
                 "cas_prefix_attn_fwd_noalloc",
                 "cas_cartridge_stage", "cas_set_tuning", "cas_get_tuning", "cas_plan_info",
                 "cas_timing_enable", "cas_timing_reset", "cas_timing_read",
                 "cas_cartridge_adam_workspace_size", "cas_cartridge_adam",
                 "cas_paged_decode_workspace_size", "cas_paged_decode_fwd", "cas_pool_plan_rotation",
                 "cas_pool_create", "cas_pool_destroy", "cas_pool_host_cartridge", "cas_pool_load",
                 "cas_pool_active", "cas_pool_end_step", "cas_pool_flush", "cas_pool_read_moments"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib
