"""ctypes declarations of libacp.so, the C ABI in include/acp.h.

Loading fails loudly when the library has not been built: there is no fallback path.
"""

from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libacp.so")

ACP_OK = 0
ACP_E_INVALID = -1
ACP_E_STEP = -2
ACP_E_STATE = -3
ACP_E_DEVICE = -4
ACP_E_UNSUPPORTED = -5
STATUS_NAMES = {0: "ACP_OK", -1: "ACP_E_INVALID", -2: "ACP_E_STEP", -3: "ACP_E_STATE",
                -4: "ACP_E_DEVICE", -5: "ACP_E_UNSUPPORTED"}

ACP_FLAG_EF = 1
ACP_FLAG_REUSE = 2
ACP_FLAG_POWERSGD = 4
ACP_FLAGS_DEFAULT = 3
ACP_FACTOR_P = 0
ACP_FACTOR_Q = 1
ACP_KERNEL_P_STEP = 1
ACP_KERNEL_Q_STEP = 2
ACP_KERNEL_Q_FINISH = 3
ACP_KERNEL_RECONSTRUCT = 4
ACP_KERNEL_ORTH = 5

_p = C.c_void_p
_i32, _i64, _u32, _u64 = C.c_int32, C.c_int64, C.c_uint32, C.c_uint64
_pi32, _pi64 = C.POINTER(C.c_int32), C.POINTER(C.c_int64)
_pf = C.c_void_p  # float* (host or device address)

# name -> (restype, argtypes), in the order of include/acp.h
SIGNATURES = {
    "acp_init": (_i32, [C.POINTER(_p), _i32, _pi32, _pi64, _i32, _u64, _i64, _i32, _u32]),
    "acp_state_bytes": (_i32, [_p, _pi64]),
    "acp_bind_state": (_i32, [_p, _p, _i64, _p]),
    "acp_num_buckets": (_i32, [_p]),
    "acp_bucket_info": (_i32, [_p, _i32, _pi32, _pi64, _pi64, _pi64]),
    "acp_layout": (_i32, [_p, _i32, _pi32, _pi64, _pi64, _pi64, _pi32]),
    "acp_tensor_info": (_i32, [_p, _i32, _pi32, _pi64, _pi64, _pi32]),
    "acp_fusion_groups": (_i32, [_p, _i32, _pi32, _pi32]),
    "acp_init_factor": (_i32, [_p, _i32, _i32, _pf, _i64]),
    "acp_compress": (_i32, [_p, _i64, _i32, _pf, _pf, _p]),
    "acp_compress_noalloc": (_i32, [_p, _i64, _i32, _pf, _pf, _p]),
    "acp_decompress": (_i32, [_p, _i64, _i32, _pf, _pf, _p]),
    "acp_compress_all": (_i32, [_p, _i64, _p, _p, _p]),
    "acp_decompress_all": (_i32, [_p, _i64, _p, _p, _p]),
    "acp_powersgd_p": (_i32, [_p, _i64, _i32, _pf, _pf, _p]),
    "acp_powersgd_q": (_i32, [_p, _i64, _i32, _pf, _pf, _pf, _p]),
    "acp_powersgd_decompress": (_i32, [_p, _i64, _i32, _pf, _pf, _p]),
    "acp_powersgd_p_all": (_i32, [_p, _i64, _p, _p, _p]),
    "acp_powersgd_q_all": (_i32, [_p, _i64, _p, _p, _p, _p]),
    "acp_powersgd_decompress_all": (_i32, [_p, _i64, _p, _p, _p]),
    "acp_error": (_i32, [_p, _i32, _pf, _p]),
    "acp_factor": (_i32, [_p, _i32, _i32, _pf, _p]),
    "acp_checkpoint_bytes": (_i32, [_p, _pi64]),
    "acp_get_state": (_i32, [_p, _p, _i64]),
    "acp_set_state": (_i32, [_p, _p, _i64]),
    "acp_profile_start": (_i32, [_p, _i32, _i32]),
    "acp_profile_stop": (_i32, [_p, _pi64, C.POINTER(C.c_double), C.POINTER(C.c_double)]),
    "acp_last_error": (C.c_char_p, [_p]),
    "acp_destroy": (None, [_p]),
}

_lib = None


class AcpError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}" + (f" ({detail})" if detail else ""))


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load libacp.so and declare its signatures (cached)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2306_08881_amd.build`")
    # torch carries its own libamdhip64.so.7; loading it first makes libacp.so bind to that
    # same HIP runtime instead of a second copy that would not know torch's devices and streams
    import torch  # noqa: F401
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib
