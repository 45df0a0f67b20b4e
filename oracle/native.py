"""Builds and loads the oracle's C part (fp8_groups.c) with gcc.

TEST INFRASTRUCTURE ONLY: part of the CPU oracle.
"""

import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "fp8_groups.c")
LIB = os.path.join(HERE, "_oracle_native.so")

_lib = None


def build() -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB)
        P = ctypes.POINTER(ctypes.c_float)
        L.fp8_conv3x3_groups.argtypes = [P, P, ctypes.c_int, ctypes.c_int, ctypes.c_int, P]
        L.fp8_conv3x3_groups.restype = None
        _lib = L
    return _lib
