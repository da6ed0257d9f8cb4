"""ctypes binding of liblacache.so (the C ABI in include/lacache.h).

Argument marshalling only: every computation runs in the library's HIP
kernels. Loading fails with an exception when the library has not been built;
there is no fallback implementation.
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblacache.so")

LACACHE_OK = 0
LACACHE_ERR_INVALID_ARG = -1
LACACHE_ERR_UNSUPPORTED = -2
LACACHE_ERR_HIP = -3
LACACHE_ERR_ALLOC = -4
LACACHE_ERR_CAPTURE = -5
LACACHE_GRAN_GROUP, LACACHE_GRAN_TOKEN, LACACHE_GRAN_TENSOR = 0, 1, 2

# name -> (restype, argtypes)
_P, _I64, _I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
SIGNATURES = {
    "lacache_quant_weights": (_I, [_P, _P, _P, _P, _I64, _I64, _I]),
    "lacache_pack_weights": (_I, [_P, _P, _P, _I64, _I64]),
    "lacache_rmsnorm_quant": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I]),
    "lacache_add_rmsnorm_quant": (_I, [_P, _P, _P, _P, _P, _P, _I64, _I64, _I]),
    "lacache_ffn_fp8_addnorm": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_gateup_swiglu_quant": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_down_proj": (_I, [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_ffn_fp8": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_ffn_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I64, _I]),
    "lacache_ffn_fp8_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_ffn_fp8_ws": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I, _P, ctypes.c_size_t]),
    "lacache_add_bf16": (_I, [_P, _P, _P, _I64]),
    "lacache_encode_e4m3": (_I, [_P, _P, _P, _I64]),
    "lacache_facache_attention": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _I64, _I]),
    "lacache_quant_weights_g": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I]),
    "lacache_rmsnorm_f32": (_I, [_P, _P, _P, _P, _I64, _I64]),
    "lacache_quant_rows_g": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I]),
    "lacache_gateup_swiglu_f32": (_I, [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_down_proj_g": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_ffn_fp8_g": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "lacache_ffn_g_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I64]),
    "lacache_embed_rmsnorm": (_I, [_P, _P, _P, _I64, _P, _I64, _P, _P, _I64, _P, _I64]),
    "lacache_linear_bf16": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64]),
    "lacache_rope_scatter": (_I, [_P, _P, _P, _I64, _P, _P, _P, _P, _P, _I64, _I64]),
    "lacache_first_layer_tokens": (_I, [_P, _P, _P, _I64, _P, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64,
                                        _I64]),
    "lacache_first_layer_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I64]),
    "lacache_set_path_policy": (_I, [_I]),
    "lacache_status_string": (ctypes.c_char_p, [_I]),
    "lacache_release_workspace": (None, []),
}

_lib = None


class LacacheError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, status_string(status), status))


def lib():
    """The loaded library (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("liblacache.so is not built (run __graft_entry__.build() or "
                               "python -m paper_2607_16339_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(status):
    return lib().lacache_status_string(int(status)).decode()


def check(status, where):
    if status != LACACHE_OK:
        raise LacacheError(status, where)
