"""ctypes binding of libknnlm.so: argument marshalling only.

Every step of the kNN-LM mixture runs in the HIP kernels behind the C ABI
declared in include/knnlm.h.  There is no fallback: if the library cannot be
loaded, importing the functions raises.
"""
from __future__ import annotations

import ctypes
import re
import sys
from typing import Dict

from . import build as _build

P = ctypes.c_void_p
I64 = ctypes.c_int64
I32 = ctypes.c_int32
I = ctypes.c_int
F = ctypes.c_float
SZ = ctypes.c_size_t

KNN_OK = 0
STATUS_NAMES = {0: "KNN_OK", 1: "KNN_ERR_INVALID_ARG", 2: "KNN_ERR_R_EXCEEDS_N", 3: "KNN_ERR_UNSUPPORTED",
                4: "KNN_ERR_WORKSPACE", 5: "KNN_ERR_HIP"}
DTYPES = {"f32": 0, "bf16": 1, "f16": 2}
KEYS_PACKED = 0x100  # OR'ed into a 16-bit dtype: the keys are the packed copy (knn_pack_keys)
PARTS = {"distances": 1, "select": 2, "mix": 3, "select_mix": 4}

_MIX_ARGS = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I64, I64, I, I32, F, F, P, P, P, P, SZ, P]
_RRC_ARGS = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I64, I64, I, I32, F, F, F, P, P, P, P, P, SZ, P]

SIGNATURES: Dict[str, tuple] = {
    "knn_lm_mixture": (I, _MIX_ARGS),
    "knn_lm_mixture_noalloc": (I, _MIX_ARGS[:22] + [P]),
    "knn_lm_mixture_rrc": (I, _RRC_ARGS),
    "knn_lm_mixture_part": (I, [I] + _MIX_ARGS),
    "knn_nest_step": (I, [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I64, I64, I, I32, F, F, F, F, P, P,
                          P, P, P, P, P, P, P, P, P, P, SZ, P]),
    "knn_spec_verify": (I, [P, P, P, P, I64, F, P, P, P, P]),
    "knn_lm_mixture_workspace_size": (SZ, [I64, I64, I64, I64, I64, I64, I64, I64, I, I32]),
    "knn_lm_mixture_validate": (I, [P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I64, I64, I, I32, F, F,
                                    P, P, P, P, SZ]),
    "knn_distances": (I, [P, P, P, P, P, I64, I64, I64, I64, I64, I, P, I64, P]),
    "knn_key_sqnorms": (I, [P, I64, I64, I, P, P]),
    "knn_pack_keys": (I, [P, I64, I64, I, P, P]),
    "knn_packed_keys_bytes": (SZ, [I64, I64, I]),
    "knn_mix": (I, [P, P, P, P, P, P, I64, I64, I64, I32, F, F, P, P]),
    "knn_mix_rrc": (I, [P, P, P, P, P, P, I64, I64, I64, I32, F, F, F, P, P, P]),
    "knn_stream_read": (I, [P, SZ, P, P]),
    "knn_status_string": (ctypes.c_char_p, [I]),
    "knn_abi_version": (I, []),
}

_lib = None


class KnnError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} returned {STATUS_NAMES.get(status, status)}: {status_string(status)}")


def library_path() -> str:
    return _build.LIB


def load() -> ctypes.CDLL:
    """Load libknnlm.so, rebuilding it first if it is missing or was built from
    other sources than the ones in the tree (a failed rebuild raises)."""
    global _lib
    if _lib is not None:
        return _lib
    if _build.stale():
        print(f"libknnlm: {_build.LIB} is missing or older than its sources; rebuilding", file=sys.stderr,
              flush=True)
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def header_functions(header_path: str) -> list:
    """Names of the functions include/knnlm.h declares."""
    text = open(header_path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*(knn_[a-z0-9_]+)\s*\(", text, flags=re.M)))


def status_string(status: int) -> str:
    return load().knn_status_string(int(status)).decode()


def check(fn: str, status: int):
    if status != KNN_OK:
        raise KnnError(fn, status)
