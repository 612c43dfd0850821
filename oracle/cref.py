"""ctypes loader for oracle/quant_ref.c -- test infrastructure only.

``build()`` compiles the C file with gcc (strict IEEE flags); ``load()`` uses
the built library, building it first only when it is missing.
"""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "quant_ref.c")
LIB = os.path.join(HERE, "liboracle_quant_ref.so")

_lib = None


def build() -> str:
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
           "-shared", "-fPIC", SRC, "-o", LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB):
        build()
    lib = ctypes.CDLL(LIB)
    P, I = ctypes.c_void_p, ctypes.c_int64
    lib.oracle_quant_weight_block128.argtypes = [P, I, I, I, P, I, P]
    lib.oracle_quant_act_token_group128.argtypes = [P, I, I, I, P, I, P, I]
    lib.oracle_e4m3_of_quotient.argtypes = [P, P, I, P]
    lib.oracle_quant_weight_block128_ue8m0.argtypes = [P, I, I, I, P, I, P]
    lib.oracle_quant_act_token_group128_ue8m0.argtypes = [P, I, I, I, P, I, P, I]
    for f in (lib.oracle_quant_weight_block128, lib.oracle_quant_act_token_group128,
              lib.oracle_e4m3_of_quotient, lib.oracle_quant_weight_block128_ue8m0,
              lib.oracle_quant_act_token_group128_ue8m0):
        f.restype = None
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def quant_weight_block128(w_bits: np.ndarray):
    w = np.ascontiguousarray(w_bits, dtype=np.uint16)
    n, k = w.shape
    if n % 128 or k % 128:
        raise ValueError("weight dims must be multiples of 128")
    q = np.empty((n, k), np.uint8)
    s = np.empty((n // 128, k // 128), np.float32)
    load().oracle_quant_weight_block128(_ptr(w), n, k, k, _ptr(q), k, _ptr(s))
    return q, s


def quant_act_token_group128(a_bits: np.ndarray, ld_scale=None):
    a = np.ascontiguousarray(a_bits, dtype=np.uint16)
    m, k = a.shape
    if k % 128:
        raise ValueError("activation K must be a multiple of 128")
    ld = m if ld_scale is None else int(ld_scale)
    q = np.empty((m, k), np.uint8)
    s = np.zeros((k // 128, ld), np.float32)
    if m:
        load().oracle_quant_act_token_group128(_ptr(a), m, k, k, _ptr(q), k, _ptr(s), ld)
    return q, s


def e4m3_of_quotient(x_bits: np.ndarray, amax_bits: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x_bits, dtype=np.uint16).ravel()
    am = np.ascontiguousarray(amax_bits, dtype=np.uint16).ravel()
    assert x.shape == am.shape
    out = np.empty(x.shape, np.uint8)
    load().oracle_e4m3_of_quotient(_ptr(x), _ptr(am), x.size, _ptr(out))
    return out


def quant_weight_block128_ue8m0(w_bits: np.ndarray):
    """Power-of-two scale variant (scales fp32 2^k)."""
    w = np.ascontiguousarray(w_bits, dtype=np.uint16)
    n, k = w.shape
    if n % 128 or k % 128:
        raise ValueError("weight dims must be multiples of 128")
    q = np.empty((n, k), np.uint8)
    s = np.empty((n // 128, k // 128), np.float32)
    load().oracle_quant_weight_block128_ue8m0(_ptr(w), n, k, k, _ptr(q), k, _ptr(s))
    return q, s


def quant_act_token_group128_ue8m0(a_bits: np.ndarray, ld_scale=None):
    """Power-of-two scale variant (scales fp32 2^k, [K/128][ld_scale], padding 0)."""
    a = np.ascontiguousarray(a_bits, dtype=np.uint16)
    m, k = a.shape
    if k % 128:
        raise ValueError("activation K must be a multiple of 128")
    ld = m if ld_scale is None else int(ld_scale)
    q = np.empty((m, k), np.uint8)
    s = np.zeros((k // 128, ld), np.float32)
    if m:
        load().oracle_quant_act_token_group128_ue8m0(_ptr(a), m, k, k, _ptr(q), k, _ptr(s), ld)
    return q, s
