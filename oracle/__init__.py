"""CPU oracle for the kNN-LM mixture step -- TEST INFRASTRUCTURE ONLY.

A plain fp64 brute force of the paper's equations (Section 2.2, eq.
non-parametric and eq. kNN-LM; Section 3.1 second-stage token search;
Appendix A), written in C (`knn_oracle.c`) and called through ctypes on host
numpy arrays.  Only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP library under
`paper_2405_19325_amd/`, and neither side imports the other.

Pinned against the paper and the mathematics by `tests/test_oracle_pins.py`:
hand-computed cases, closed forms (sum of p_M, lambda = 1 and 0, r = 1,
duplicate tokens, mu -> 0), a textbook softmax when r = N, a stable argsort on
tiny inputs, exact-integer inputs, metamorphic invariances, and the element
decoding against numpy / torch conversions; relative retrieval confidence
(Section 3.2, eq. rrc) by sigmoid values known in closed form, its symmetry,
its scale invariance and a hand-worked case.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "knn_oracle.c")
_LIB = os.path.join(_HERE, "libknn_oracle.so")

DTYPE_CODES = {"f32": 0, "bf16": 1, "f16": 2}

_lib = None


def build() -> str:
    """Compile the oracle with gcc (plain C, no GPU code)."""
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC", "-pthread", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P, I64, I32, I, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int, ctypes.c_double
    lib.knn_oracle_widen.argtypes = [P, I, I64, P]
    lib.knn_oracle_sqdist.argtypes = [P, P, I, I64, I64, I64, I, P]
    lib.knn_oracle_select.argtypes = [P, P, I, I64, I64, P, P, I64, I32, I, P, P]
    lib.knn_oracle_select_masked.argtypes = [P, P, I, I64, I64, P, P, I64, I32, P, I, P, P]
    lib.knn_oracle_mix.argtypes = [P, P, P, P, P, I64, I64, I32, P, I64, D, D, P, P]
    lib.knn_oracle_mix_lambdas.argtypes = [P, P, P, P, P, I64, I64, I32, P, I64, D, P, P, P]
    lib.knn_oracle_rrc_lambda.argtypes = [P, I64, I32, D, D, P]
    for f in (lib.knn_oracle_widen, lib.knn_oracle_sqdist, lib.knn_oracle_select, lib.knn_oracle_mix):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} rejected its arguments (code {rc})")


def _raw(a: np.ndarray) -> np.ndarray:
    """Element bytes of a host array as a C-contiguous uint8/uint16/float32 view."""
    return np.ascontiguousarray(a)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def widen(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Decode stored elements (float32 values, or uint16 bit patterns) to fp64."""
    raw = _raw(raw)
    out = np.empty(raw.size, dtype=np.float64)
    _check(_load().knn_oracle_widen(_ptr(raw), DTYPE_CODES[dtype], raw.size, _ptr(out)), "widen")
    return out.reshape(raw.shape)


def sqdist(queries: np.ndarray, keys: np.ndarray, dtype: str, nthreads: Optional[int] = None) -> np.ndarray:
    """All fp64 squared distances [nq, nk] (direct sum of squared differences)."""
    queries, keys = _raw(queries), _raw(keys)
    nq, d = queries.shape
    nk = keys.shape[0]
    assert keys.shape[1] == d
    out = np.empty((nq, nk), dtype=np.float64)
    _check(_load().knn_oracle_sqdist(_ptr(queries), _ptr(keys), DTYPE_CODES[dtype], nq, nk, d,
                                     nthreads or default_threads(), _ptr(out)), "sqdist")
    return out


def select(queries: np.ndarray, keys: np.ndarray, dtype: str, key_offsets: np.ndarray,
           query_offsets: np.ndarray, r: int, nthreads: Optional[int] = None,
           key_mask: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Per query: the r nearest local key ids of its own set, ascending by (dist, id), and their dists.

    key_mask: uint32 words, bit (i & 31) of word i >> 5 set for a masked global key row i
    (Section 3.4); masked keys are never neighbours, and slots the unmasked keys cannot
    fill hold id -1 and distance +inf."""
    queries, keys = _raw(queries), _raw(keys)
    ko = np.ascontiguousarray(key_offsets, dtype=np.int64)
    qo = np.ascontiguousarray(query_offsets, dtype=np.int64)
    B, d = queries.shape
    ids = np.empty((B, r), dtype=np.int32)
    dists = np.empty((B, r), dtype=np.float64)
    mask = None if key_mask is None else np.ascontiguousarray(key_mask, dtype=np.uint32)
    if mask is not None and mask.size * 32 < int(ko[-1]):
        raise ValueError("key_mask needs one bit per key row")
    rc = _load().knn_oracle_select_masked(_ptr(queries), _ptr(keys), DTYPE_CODES[dtype], B, d, _ptr(ko), _ptr(qo),
                                          len(ko) - 1, r, _ptr(mask), nthreads or default_threads(), _ptr(ids),
                                          _ptr(dists))
    _check(rc, "select")
    return ids, dists


def mix(ids: np.ndarray, dists: np.ndarray, values: np.ndarray, key_offsets: np.ndarray,
        query_offsets: np.ndarray, p_lm: np.ndarray, mu: float, lam,
        want_pknn: bool = False):
    """p_M (and optionally p_kNN) in fp64 from per-query neighbour ids and fp64 distances.

    `lam` is one weight of p_LM for every query (eq. kNN-LM) or an array of
    one weight per query (e.g. from rrc_lambda)."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    dists = np.ascontiguousarray(dists, dtype=np.float64)
    values = np.ascontiguousarray(values, dtype=np.int32)
    ko = np.ascontiguousarray(key_offsets, dtype=np.int64)
    qo = np.ascontiguousarray(query_offsets, dtype=np.int64)
    p_lm = np.ascontiguousarray(p_lm, dtype=np.float32)
    B, r = ids.shape
    V = p_lm.shape[1]
    pm = np.empty((B, V), dtype=np.float64)
    pk = np.empty((B, V), dtype=np.float64) if want_pknn else None
    if np.ndim(lam) == 0:
        rc = _load().knn_oracle_mix(_ptr(ids), _ptr(dists), _ptr(values), _ptr(ko), _ptr(qo), len(ko) - 1, B, r,
                                    _ptr(p_lm), V, float(mu), float(lam), _ptr(pm), _ptr(pk))
    else:
        lams = np.ascontiguousarray(lam, dtype=np.float64)
        if lams.shape != (B,):
            raise ValueError("one lambda per query")
        rc = _load().knn_oracle_mix_lambdas(_ptr(ids), _ptr(dists), _ptr(values), _ptr(ko), _ptr(qo), len(ko) - 1,
                                            B, r, _ptr(p_lm), V, float(mu), _ptr(lams), _ptr(pm), _ptr(pk))
    _check(rc, "mix")
    return (pm, pk) if want_pknn else pm


def rrc_lambda(dists: np.ndarray, alpha: float, tau: float) -> np.ndarray:
    """Per-query lambda_t of relative retrieval confidence (Section 3.2, eq. rrc) from each
    query's r neighbour distances (any order), in fp64."""
    dists = np.ascontiguousarray(dists, dtype=np.float64)
    B, r = dists.shape
    out = np.empty(B, dtype=np.float64)
    _check(_load().knn_oracle_rrc_lambda(_ptr(dists), B, r, float(alpha), float(tau), _ptr(out)), "rrc_lambda")
    return out


def host_elements(t) -> Tuple[np.ndarray, str]:
    """Stored bytes of a torch tensor as a host numpy array the oracle reads, plus its dtype code name."""
    import torch

    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.float32:
        return t.numpy(), "f32"
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16), "bf16"
    if t.dtype == torch.float16:
        return t.view(torch.int16).numpy().view(np.uint16), "f16"
    raise TypeError(t.dtype)


def run(workload, nthreads: Optional[int] = None, want_pknn: bool = False):
    """The whole step on a workload's inputs (copied to host): ids, fp64 dists, fp64 p_M."""
    q, dt = host_elements(workload.queries)
    k, _ = host_elements(workload.keys)
    ids, dists = select(q, k, dt, workload.key_offsets_host, workload.query_offsets_host, workload.r, nthreads)
    vals = workload.values.to("cpu").numpy()
    p_lm = workload.p_lm.to("cpu").numpy()
    out = mix(ids, dists, vals, workload.key_offsets_host, workload.query_offsets_host, p_lm,
              workload.mu, workload.lam, want_pknn=want_pknn)
    if want_pknn:
        return ids, dists, out[0], out[1]
    return ids, dists, out
