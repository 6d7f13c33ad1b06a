"""ctypes binding of libmiriam.so (the C ABI declared in include/miriam.h).

Argument marshalling only: every entry point keeps its C name and signature.
The library is loaded from this package's directory; if it is missing the
import fails loudly (there is no CPU fallback of any kernel).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmiriam.so")

# ---------------------------------------------------------------- enums
OK, EINVAL, ERANGE, EHIP, ENOMEM, EBUSY, ESTATE, ENOTFOUND = 0, -1, -2, -3, -4, -5, -6, -7
ERR_NAMES = {0: "OK", -1: "EINVAL", -2: "ERANGE", -3: "EHIP", -4: "ENOMEM", -5: "EBUSY",
             -6: "ESTATE", -7: "ENOTFOUND"}

OP_CONV2D, OP_GEMM, OP_BGEMM, OP_DWCONV, OP_POOL_MAX, OP_POOL_AVG, OP_SOFTMAX, OP_LAYERNORM, OP_BN_ACT = range(9)
F32, F16, BF16 = 0, 1, 2
DTYPE_CODE = {"f32": F32, "f16": F16, "bf16": BF16}
ACT_NONE, ACT_RELU, ACT_RELU6, ACT_GELU = 0, 1, 2, 3
ACT_CODE = {"none": 0, "relu": 1, "relu6": 2, "gelu": 3}
EPI_BIAS, EPI_BN, EPI_RESIDUAL = 1, 2, 4
INDEX_MEMORY = 8  # memory-based index function (host-computed row table)
POLICY_ELASTIC, POLICY_SEQUENTIAL, POLICY_MULTISTREAM, POLICY_IB = 0, 1, 2, 3
BACKEND_HIP, BACKEND_FAKE = 0, 1


class OpDesc(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("act", ctypes.c_int32),
        ("flags", ctypes.c_int32),
        ("n", ctypes.c_int64), ("h", ctypes.c_int64), ("w", ctypes.c_int64), ("c", ctypes.c_int64),
        ("k", ctypes.c_int64),
        ("kh", ctypes.c_int64), ("kw", ctypes.c_int64), ("stride", ctypes.c_int64),
        ("pad", ctypes.c_int64), ("groups", ctypes.c_int64),
        ("m", ctypes.c_int64), ("nn", ctypes.c_int64), ("kk", ctypes.c_int64),
        ("batch", ctypes.c_int64), ("batch_div", ctypes.c_int64),
        ("ldx", ctypes.c_int64), ("ldw", ctypes.c_int64), ("ldy", ctypes.c_int64),
        ("sx0", ctypes.c_int64), ("sx1", ctypes.c_int64), ("sw0", ctypes.c_int64),
        ("sw1", ctypes.c_int64), ("sy0", ctypes.c_int64), ("sy1", ctypes.c_int64),
        ("b_nmajor", ctypes.c_int32), ("ksplit", ctypes.c_int32), ("tile", ctypes.c_int32),
        ("eps", ctypes.c_float), ("scale", ctypes.c_float),
        ("x", ctypes.c_void_p), ("wt", ctypes.c_void_p), ("bias", ctypes.c_void_p),
        ("bn", ctypes.c_void_p), ("residual", ctypes.c_void_p), ("y", ctypes.c_void_p),
    ]


class OpInfo(ctypes.Structure):
    _fields_ = [
        ("num_tiles", ctypes.c_int64), ("logical_block", ctypes.c_int32),
        ("lds_bytes", ctypes.c_int32), ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
        ("max_wg_per_cu", ctypes.c_int32 * 3), ("flops", ctypes.c_double), ("bytes", ctypes.c_double),
        ("path", ctypes.c_int32), ("ksplit", ctypes.c_int32), ("full_grid", ctypes.c_int32),
    ]


# miriam_kernel_path
PATH_OTHER, PATH_STAGED, PATH_DMA, PATH_DMA_UNIFORM, PATH_SKINNY, PATH_HALO, PATH_RESIDENT = 0, 1, 2, 3, 4, 5, 6


class DeviceDesc(ctypes.Structure):
    _fields_ = [
        ("n_cu", ctypes.c_int32), ("max_threads_per_cu", ctypes.c_int32),
        ("lds_per_cu", ctypes.c_int32), ("n_xcd", ctypes.c_int32), ("wave_size", ctypes.c_int32),
        ("clock_khz", ctypes.c_int32), ("arch", ctypes.c_char * 64),
    ]


class Config(ctypes.Structure):
    _fields_ = [
        ("policy", ctypes.c_int32), ("backend", ctypes.c_int32), ("n_be_streams", ctypes.c_int32),
        ("inflight_depth", ctypes.c_int32), ("top_frac", ctypes.c_double),
        ("max_blk_frac", ctypes.c_double), ("max_pt_frac", ctypes.c_double),
        ("quantum_us", ctypes.c_double), ("inflight_us", ctypes.c_double),
        ("busy_policy", ctypes.c_int32),
        ("log_launches", ctypes.c_int32), ("profile_reps", ctypes.c_int32),
        ("fake_n_cu", ctypes.c_int32), ("fake_slots_per_cu", ctypes.c_int32),
        ("fake_tile_ns", ctypes.c_double), ("fake_launch_ns", ctypes.c_double),
        ("graphs", ctypes.c_int32), ("release_guard", ctypes.c_int32), ("warm_critical", ctypes.c_int32),
        ("graph_chunk", ctypes.c_int32), ("arm_lead_us", ctypes.c_double),
        ("segments", ctypes.c_int32), ("event_us", ctypes.c_double),
        ("be_cu_reserve", ctypes.c_int32), ("whole_when_clear", ctypes.c_int32),
        ("whole_margin", ctypes.c_double), ("fake_fail_launch", ctypes.c_int32),
        ("crit_cu_exclusive", ctypes.c_int32),
    ]


class LaunchRecord(ctypes.Structure):
    _fields_ = [
        ("ticket", ctypes.c_uint64), ("op_index", ctypes.c_int32), ("stream", ctypes.c_int32),
        ("criticality", ctypes.c_int32), ("grid", ctypes.c_int32), ("block", ctypes.c_int32),
        ("crit_busy", ctypes.c_int32), ("shard_begin", ctypes.c_int64), ("shard_len", ctypes.c_int64),
        ("num_tiles", ctypes.c_int64), ("eq2_grid_limit", ctypes.c_int64), ("t_issue_ns", ctypes.c_int64),
        ("est_us", ctypes.c_double),
    ]


class Completion(ctypes.Structure):
    _fields_ = [
        ("ticket", ctypes.c_uint64), ("criticality", ctypes.c_int32), ("status", ctypes.c_int32),
        ("t_release_ns", ctypes.c_int64), ("t_start_ns", ctypes.c_int64), ("t_end_ns", ctypes.c_int64),
        ("deadline_ns", ctypes.c_int64), ("deadline_met", ctypes.c_int32), ("n_shards", ctypes.c_int32),
    ]


class Stats(ctypes.Structure):
    _fields_ = [
        ("launches", ctypes.c_int64), ("shards_sized", ctypes.c_int64),
        ("eq2_violations", ctypes.c_int64), ("decisions", ctypes.c_int64),
        ("decision_ns_total", ctypes.c_double), ("completed", ctypes.c_int64),
        ("graph_launches", ctypes.c_int64), ("warm_launches", ctypes.c_int64),
        ("armed_releases", ctypes.c_int64), ("segment_launches", ctypes.c_int64),
        ("barrier_groups", ctypes.c_int64), ("whole_clear_launches", ctypes.c_int64),
        ("failed_requests", ctypes.c_int64), ("failed_pass_resets", ctypes.c_int64),
    ]


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32P = ctypes.POINTER(ctypes.c_int32)
_I64P = ctypes.POINTER(ctypes.c_int64)
_DP = ctypes.POINTER(ctypes.c_double)
_INT = ctypes.c_int

SIGNATURES = {
    "miriam_last_error": ([], ctypes.c_char_p),
    "miriam_device_query": ([ctypes.POINTER(DeviceDesc)], _INT),
    "miriam_op_create": ([ctypes.POINTER(OpDesc), ctypes.POINTER(_P)], _INT),
    "miriam_op_create_noalloc": ([ctypes.POINTER(OpDesc), ctypes.POINTER(_P)], _INT),
    "miriam_op_query": ([_P, ctypes.POINTER(OpInfo)], _INT),
    "miriam_elastic_launch": ([_P, _I64, _I64, _INT, _INT, _P], _INT),
    "miriam_elastic_launch_traced": ([_P, _I64, _I64, _INT, _INT, _P, _P, _P, _P, _P, _P], _INT),
    "miriam_op_destroy": ([_P], _INT),
    "miriam_op_reset_counters": ([_P, _P], _INT),
    "miriam_plan_dichotomy": ([_I64, _I64P, _INT], _INT),
    "miriam_plan_split": ([_I64, _I64, _I64P, _I64P], _INT),
    "miriam_plan_wg_rank": ([_I64, _I64, _I64], _I64),
    "miriam_plan_eq2_grid_limit": ([_I64, _I64], _I64),
    "miriam_plan_eq2_block_limit": ([_I64, _I64], _I64),
    "miriam_plan_wiscore": ([_I64] * 6, ctypes.c_double),
    "miriam_plan_oscore": ([_I64, _DP, _DP, ctypes.c_double, ctypes.c_double], _INT),
    "miriam_plan_top_fraction": ([_INT, _DP, _I64P, _I64P, ctypes.c_double,
                                  ctypes.POINTER(_INT)], _INT),
    "miriam_plan_tree_head": ([_I64, _I64, _I64, ctypes.POINTER(_INT)], _I64),
    "miriam_init": ([ctypes.POINTER(Config)], _INT),
    "miriam_task_create": ([ctypes.POINTER(_P), _INT, ctypes.POINTER(_P)], _INT),
    "miriam_submit": ([_P, _INT, _I64, _I64, ctypes.POINTER(ctypes.c_uint64)], _INT),
    "miriam_poll": ([ctypes.POINTER(Completion), _INT], _INT),
    "miriam_drain": ([_I64], _INT),
    "miriam_stats_get": ([ctypes.POINTER(Stats)], _INT),
    "miriam_task_destroy": ([_P], _INT),
    "miriam_shutdown": ([], _INT),
    "miriam_now_ns": ([], _I64),
    "miriam_launch_log": ([ctypes.POINTER(LaunchRecord), _INT], _INT),
    "miriam_gate_check": ([_P, _I64, _I64, _DP], _INT),
}

_lib = None


def load():
    """Load libmiriam.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2307_04339_amd.build` "
            "(there is no fallback implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (args, res) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


class MiriamError(RuntimeError):
    def __init__(self, rc: int, what: str):
        self.rc = rc
        msg = load().miriam_last_error().decode(errors="replace")
        super().__init__(f"{what}: {ERR_NAMES.get(rc, rc)} ({msg})")


def check(rc: int, what: str) -> int:
    if rc < 0:
        raise MiriamError(rc, what)
    return rc
