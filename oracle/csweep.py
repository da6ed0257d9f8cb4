"""ctypes wrapper of oracle/e4m3_sweep.c (oracle; test infrastructure only).

The shared object is compiled by ``build_csweep()`` with gcc into this
directory. It serves exhaustive sweeps of the e4m3 encoder over fp32 bit
patterns, where the NumPy encoder would be too slow.
"""

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "e4m3_sweep.c")
_LIB = os.path.join(_HERE, "libe4m3sweep.so")
_lib = None


def build_csweep():
    """Compile e4m3_sweep.c with gcc (always recompiles)."""
    cmd = ["gcc", "-O2", "-std=c11", "-shared", "-fPIC", _SRC, "-o", _LIB, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build_csweep()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_e4m3_encode_f32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        lib.oracle_e4m3_encode_f32.restype = None
        lib.oracle_e4m3_sweep_check.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.c_int64,
                                                ctypes.POINTER(ctypes.c_uint32)]
        lib.oracle_e4m3_sweep_check.restype = ctypes.c_int64
        _lib = lib
    return _lib


def encode_f32(v):
    """Encode a float32 array with the C encoder; returns uint8 codes."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(v.shape, dtype=np.uint8)
    _load().oracle_e4m3_encode_f32(v.ctypes.data, out.ctypes.data, v.size)
    return out


def sweep_check(codes, first_bits):
    """Compare codes for the fp32 patterns first_bits .. first_bits+len-1.

    Returns (mismatch_count, first_bad_bits or None); non-finite inputs skipped.
    """
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    fb = ctypes.c_uint32(0)
    n = _load().oracle_e4m3_sweep_check(codes.ctypes.data, ctypes.c_uint32(first_bits), codes.size,
                                        ctypes.byref(fb))
    return int(n), (int(fb.value) if n else None)
