"""ctypes binding of libmoeshard.so: the C ABI declared in include/moeshard.h.

Loading fails loudly if the library has not been built; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import threading

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoeshard.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP, MOE_ERR_TOO_LARGE = range(6)
MOE_NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024
MOE_F32, MOE_BF16 = 0, 1
MOE_ACT_GELU, MOE_ACT_GELU_TANH, MOE_ACT_SWIGLU = 0, 1, 2
MOE_MAX_EXPERTS = 256

ACTS = {"gelu": MOE_ACT_GELU, "gelu_tanh": MOE_ACT_GELU_TANH, "swiglu": MOE_ACT_SWIGLU}

# name -> (restype, argtypes)
_P, _I64, _I32, _SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
_ST = ctypes.c_int
SIGNATURES = {
    "moe_status_string": (ctypes.c_char_p, [_ST]),
    "moe_route": (_ST, [_P, _ST, _I64, _I64, _P, _I32, _I32, _P, _I64, _I32, _P, _P, _P]),
    "moe_dispatch_workspace_size": (_SZ, [_I64, _I32, _I32]),
    "moe_route_dispatch": (_ST, [_P, _ST, _I64, _I64, _P, _I32, _I32, _P, _I64, _I32, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                 _P]),
    "moe_dispatch": (_ST, [_P, _I64, _I32, _I32, _P, _ST, _I64, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "moe_padded_inner_width": (_I64, [_I64]),
    "moe_packed_weights_size": (_SZ, [_I32, _I64, _I64, _ST, _ST]),
    "moe_pack_weights": (_ST, [_P, _P, _P, _I32, _I64, _I64, _I64, _I64, _ST, _ST, _P, _SZ, _P]),
    "moe_ffn_workspace_size": (_SZ, [_I64, _I32, _I64, _I64, _ST, _ST]),
    "moe_expert_ffn_shard": (_ST, [_P, _P, _I64, _I32, _I64, _I64, _ST, _ST, _P, _P, _ST, _P, _SZ, _P]),
    "moe_expert_ffn_shard_gather": (_ST, [_P, _I64, _P, _P, _I64, _I32, _I64, _I64, _ST, _ST, _P, _P, _ST, _P, _SZ,
                                          _P]),
    "moe_expert_ffn_shard_gather_combine": (_ST, [_P, _I64, _P, _P, _P, _P, _I32, _I32, _I64, _I64, _ST, _ST, _P, _P,
                                                  _ST, _P, _ST, _P, _P, _SZ, _P]),
    "moe_expert_ffn_shard_top1": (_ST, [_P, _I64, _P, _P, _P, _I32, _I64, _I64, _ST, _ST, _P, _P, _ST, _P, _SZ, _P]),
    "moe_expert_ffn_shard_per_expert": (_ST, [_P, _P, _P, _I64, _I32, _I64, _I64, _ST, _ST, _P, _P, _ST, _P, _SZ,
                                              _P]),
    "moe_expert_ffn_shard_noalloc": (_ST, [_P, _P, _I64, _I32, _I64, _I64, _ST, _ST, _P, _P, _ST, _P]),
    "moe_combine": (_ST, [_P, _ST, _P, _P, _I64, _I32, _I64, _P, _ST, _P]),
}

_lock = threading.Lock()
_lib = None


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {status_string(status)}")


def load() -> ctypes.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2503_08467_amd.build` "
                    "(there is no CPU fallback)")
            lib = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def status_string(status: int) -> str:
    return load().moe_status_string(status).decode()


def call(name: str, *args) -> None:
    st = getattr(load(), name)(*args)
    if st != MOE_OK:
        raise MoeError(name, st)
