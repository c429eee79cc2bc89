"""MI355X-native kNN-LM mixture step (Nearest Neighbor Speculative Decoding, Section 2.2).

The Python surface mirrors the C ABI in include/knnlm.h and only marshals
arguments: device tensors are passed as raw pointers together with the
current torch stream.  All arithmetic runs in the HIP kernels of libknnlm.so.

    prob = MixtureProblem(queries, keys, values, key_offsets, query_offsets, p_lm, r, mu, lam)
    p_m, ids, dists = prob.run()
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np
import torch

from . import _lib
from ._lib import DTYPES, KEYS_PACKED, PARTS, KnnError, load, status_string  # noqa: F401

__all__ = ["MixtureProblem", "mixture", "mixture_noalloc", "distances", "key_sqnorms", "pack_keys",
           "packed_keys_bytes", "mix", "mix_rrc", "spec_verify", "mask_words", "stream_read", "workspace_size",
           "KnnError", "load", "status_string", "abi_version"]

_TORCH_DTYPES = {torch.float32: "f32", torch.bfloat16: "bf16", torch.float16: "f16"}


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _dtype_code(t: torch.Tensor) -> int:
    try:
        return DTYPES[_TORCH_DTYPES[t.dtype]]
    except KeyError:
        raise TypeError(f"unsupported element type {t.dtype}") from None


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def abi_version() -> int:
    return load().knn_abi_version()


def workspace_size(B, d, V, S, total_keys, min_keys, max_keys, max_queries, dtype: str, r) -> int:
    return int(load().knn_lm_mixture_workspace_size(B, d, V, S, total_keys, min_keys, max_keys, max_queries,
                                                    DTYPES[dtype], r))


class MixtureProblem:
    """Inputs, planning hints, workspace and outputs of repeated knn_lm_mixture calls.

    queries [B, d], keys [total_keys, d] (same dtype: f32/bf16/f16), values
    [total_keys] int32, key_offsets / query_offsets [S+1] int64, p_lm [B, V]
    fp32, all on one GPU.  The host copies of the offsets (derived once here
    unless given) provide the planning hints.  packed_keys, the packed copy of
    `keys` from pack_keys(), makes the distance stage read that copy instead
    (query batches on the matrix cores only; the results are the same bits).
    """

    def __init__(self, queries: torch.Tensor, keys: torch.Tensor, values: torch.Tensor,
                 key_offsets: torch.Tensor, query_offsets: torch.Tensor, p_lm: torch.Tensor, r: int,
                 mu: Optional[float] = None, lam: float = 0.3, key_sqnorms: Optional[torch.Tensor] = None,
                 key_offsets_host: Optional[Sequence[int]] = None,
                 query_offsets_host: Optional[Sequence[int]] = None, packed_keys: Optional[torch.Tensor] = None):
        _need(queries.dim() == 2 and keys.dim() == 2, "queries and keys must be 2-D")
        _need(queries.dtype == keys.dtype, "queries must carry the key element type")
        _need(queries.shape[1] == keys.shape[1], "queries and keys must have the same width")
        for name, t in (("queries", queries), ("keys", keys), ("values", values), ("p_lm", p_lm),
                        ("key_offsets", key_offsets), ("query_offsets", query_offsets)):
            _need(t.is_cuda, f"{name} must be a device tensor")
            _need(t.is_contiguous(), f"{name} must be contiguous")
        _need(values.dtype == torch.int32 and p_lm.dtype == torch.float32, "values int32, p_lm float32")
        _need(key_offsets.dtype == torch.int64 and query_offsets.dtype == torch.int64, "offsets must be int64")
        ko = np.asarray(key_offsets_host if key_offsets_host is not None else key_offsets.cpu().numpy(), np.int64)
        qo = np.asarray(query_offsets_host if query_offsets_host is not None else query_offsets.cpu().numpy(),
                        np.int64)
        _need(len(ko) == len(qo) and len(ko) >= 2, "offsets must have S+1 >= 2 entries")
        nk = np.diff(ko)
        nq = np.diff(qo)
        self.queries, self.keys, self.values = queries, keys, values
        self.key_offsets, self.query_offsets, self.p_lm = key_offsets, query_offsets, p_lm
        self.key_sqnorms = key_sqnorms
        self.B, self.d = int(queries.shape[0]), int(queries.shape[1])
        self.V = int(p_lm.shape[1])
        self.S = len(ko) - 1
        self.total_keys = int(keys.shape[0])
        self.min_keys = int(nk[nq > 0].min()) if (nq > 0).any() else 0
        self.max_keys = int(nk.max())
        self.max_queries = int(nq.max())
        self.dtype = _dtype_code(queries)
        self.packed_keys = packed_keys
        self.keys_arg = keys  # what the distance stage reads
        if packed_keys is not None:
            want = packed_keys_bytes(self.total_keys, self.d, keys.dtype)
            _need(packed_keys.is_cuda and packed_keys.is_contiguous() and
                  packed_keys.numel() * packed_keys.element_size() == want,
                  f"packed_keys: the {want}-byte packed copy of keys (pack_keys)")
            self.keys_arg = packed_keys
            self.dtype |= KEYS_PACKED
        self.r = int(r)
        self.mu = float(1.0 / math.sqrt(self.d) if mu is None else mu)
        self.lam = float(lam)
        dev = queries.device
        nbytes = load().knn_lm_mixture_workspace_size(self.B, self.d, self.V, self.S, self.total_keys,
                                                      self.min_keys, self.max_keys, self.max_queries,
                                                      self.dtype, self.r)
        if nbytes == 0:
            _lib.check("knn_lm_mixture_workspace_size", self._validate(None, 0))
        self.workspace = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=dev)
        self.p_m = torch.empty((self.B, self.V), dtype=torch.float32, device=dev)
        self.ids = torch.empty((self.B, self.r), dtype=torch.int32, device=dev)
        self.dists = torch.empty((self.B, self.r), dtype=torch.float32, device=dev)
        self.lambdas = torch.empty(self.B, dtype=torch.float32, device=dev)  # lambda_t of run_rrc

    def _args(self, stream):
        return (_ptr(self.queries), _ptr(self.keys_arg), _ptr(self.key_sqnorms), _ptr(self.values),
                _ptr(self.key_offsets), _ptr(self.query_offsets), _ptr(self.p_lm), self.B, self.d, self.V, self.S,
                self.total_keys, self.min_keys, self.max_keys, self.max_queries, self.dtype, self.r, self.mu,
                self.lam, _ptr(self.p_m), _ptr(self.ids), _ptr(self.dists), _ptr(self.workspace),
                self.workspace.numel(), _stream(stream))

    def _validate(self, ws, ws_bytes):
        return load().knn_lm_mixture_validate(
            _ptr(self.queries), _ptr(self.keys_arg), _ptr(self.values), _ptr(self.key_offsets), _ptr(self.query_offsets),
            _ptr(self.p_lm), self.B, self.d, self.V, self.S, self.total_keys, self.min_keys, self.max_keys,
            self.max_queries, self.dtype, self.r, self.mu, self.lam, 1, 1, 1, ws, ws_bytes)

    def run(self, stream=None):
        """One knn_lm_mixture call; returns (p_m, nbr_ids, nbr_dists), valid after stream sync."""
        _lib.check("knn_lm_mixture", load().knn_lm_mixture(*self._args(stream)))
        return self.p_m, self.ids, self.dists

    def run_rrc(self, alpha: float, tau: float, stream=None):
        """One knn_lm_mixture_rrc call (lambda_t per query from relative retrieval
        confidence); returns (p_m, nbr_ids, nbr_dists, lambda_t [B]), valid after stream sync."""
        st = load().knn_lm_mixture_rrc(
            _ptr(self.queries), _ptr(self.keys_arg), _ptr(self.key_sqnorms), _ptr(self.values), _ptr(self.key_offsets),
            _ptr(self.query_offsets), _ptr(self.p_lm), self.B, self.d, self.V, self.S, self.total_keys,
            self.min_keys, self.max_keys, self.max_queries, self.dtype, self.r, self.mu, float(alpha), float(tau),
            _ptr(self.lambdas), _ptr(self.p_m), _ptr(self.ids), _ptr(self.dists), _ptr(self.workspace),
            self.workspace.numel(), _stream(stream))
        _lib.check("knn_lm_mixture_rrc", st)
        return self.p_m, self.ids, self.dists, self.lambdas

    def run_nest(self, alpha: float, tau: float, delta: float, key_mask: Optional[torch.Tensor] = None,
                 draft_tokens: Optional[torch.Tensor] = None, stream=None) -> dict:
        """One knn_nest_step call: the RRC mixture with masked keys left out and the step's
        decoding outputs.  Returns a dict of device tensors: p_m, ids, dists, lambdas,
        next_token, p_max, span_key, use_span and (with draft_tokens) p_draft."""
        if not hasattr(self, "next_token"):
            dev = self.p_m.device
            self.next_token = torch.empty(self.B, dtype=torch.int32, device=dev)
            self.p_max = torch.empty(self.B, dtype=torch.float32, device=dev)
            self.p_draft = torch.empty(self.B, dtype=torch.float32, device=dev)
            self.span_key = torch.empty(self.B, dtype=torch.int32, device=dev)
            self.use_span = torch.empty(self.B, dtype=torch.int32, device=dev)
        if key_mask is not None:
            _need(key_mask.is_cuda and key_mask.dtype == torch.int32 and key_mask.is_contiguous(),
                  "key_mask: contiguous int32 device words (see mask_words)")
            _need(key_mask.numel() * 32 >= self.total_keys, "key_mask needs one bit per key row")
        if draft_tokens is not None:
            _need(draft_tokens.is_cuda and draft_tokens.dtype == torch.int32 and draft_tokens.numel() == self.B,
                  "draft_tokens: [B] int32 device tensor")
        st = load().knn_nest_step(
            _ptr(self.queries), _ptr(self.keys_arg), _ptr(self.key_sqnorms), _ptr(self.values), _ptr(self.key_offsets),
            _ptr(self.query_offsets), _ptr(self.p_lm), self.B, self.d, self.V, self.S, self.total_keys,
            self.min_keys, self.max_keys, self.max_queries, self.dtype, self.r, self.mu, float(alpha), float(tau),
            float(delta), _ptr(key_mask), _ptr(draft_tokens), _ptr(self.lambdas), _ptr(self.p_m), _ptr(self.ids),
            _ptr(self.dists), _ptr(self.next_token), _ptr(self.p_max),
            _ptr(self.p_draft) if draft_tokens is not None else None, _ptr(self.span_key), _ptr(self.use_span),
            _ptr(self.workspace), self.workspace.numel(), _stream(stream))
        _lib.check("knn_nest_step", st)
        out = {"p_m": self.p_m, "ids": self.ids, "dists": self.dists, "lambdas": self.lambdas,
               "next_token": self.next_token, "p_max": self.p_max, "span_key": self.span_key,
               "use_span": self.use_span}
        if draft_tokens is not None:
            out["p_draft"] = self.p_draft
        return out

    def run_part(self, part: str, stream=None):
        """One stage ("distances", "select", "mix", "select_mix") of knn_lm_mixture on this problem's workspace."""
        _lib.check("knn_lm_mixture_part", load().knn_lm_mixture_part(PARTS[part], *self._args(stream)))


def mixture(queries, keys, values, key_offsets, query_offsets, p_lm, r, mu=None, lam=0.3, key_sqnorms=None,
            key_offsets_host=None, query_offsets_host=None):
    """One-shot knn_lm_mixture: returns (p_m [B,V] fp32, ids [B,r] int32, dists [B,r] fp32)."""
    prob = MixtureProblem(queries, keys, values, key_offsets, query_offsets, p_lm, r, mu, lam, key_sqnorms,
                          key_offsets_host, query_offsets_host)
    return prob.run()


def mixture_noalloc(queries, keys, values, key_offsets, query_offsets, p_lm, r, mu, lam, p_m, ids, dists,
                    key_offsets_host, query_offsets_host, key_sqnorms=None, stream=None):
    """knn_lm_mixture_noalloc: the step into the caller's p_m [B, V] fp32, ids [B, r] int32 and
    dists [B, r] fp32, with the library's static per-GPU scratch array as workspace (nothing
    is allocated; the host offsets give the planning hints)."""
    ko = np.asarray(key_offsets_host, np.int64)
    qo = np.asarray(query_offsets_host, np.int64)
    nk, nq = np.diff(ko), np.diff(qo)
    B, d = int(queries.shape[0]), int(queries.shape[1])
    V = int(p_lm.shape[1])
    min_keys = int(nk[nq > 0].min()) if (nq > 0).any() else 0
    for name, t, dt, shape in (("p_m", p_m, torch.float32, (B, V)), ("ids", ids, torch.int32, (B, r)),
                               ("dists", dists, torch.float32, (B, r))):
        _need(t.is_cuda and t.dtype == dt and t.is_contiguous() and tuple(t.shape) == shape,
              f"{name}: contiguous {tuple(shape)} {dt} device tensor")
    st = load().knn_lm_mixture_noalloc(
        _ptr(queries), _ptr(keys), _ptr(key_sqnorms), _ptr(values), _ptr(key_offsets), _ptr(query_offsets),
        _ptr(p_lm), B, d, V, len(ko) - 1, int(keys.shape[0]), min_keys, int(nk.max()), int(nq.max()),
        _dtype_code(queries), int(r), float(1.0 / math.sqrt(d) if mu is None else mu), float(lam), _ptr(p_m),
        _ptr(ids), _ptr(dists), _stream(stream))
    _lib.check("knn_lm_mixture_noalloc", st)
    return p_m, ids, dists


def distances(queries, keys, key_offsets, query_offsets, key_sqnorms=None, key_offsets_host=None,
              query_offsets_host=None, ld: Optional[int] = None, packed_keys: Optional[torch.Tensor] = None):
    """knn_distances: squared distances [B, ld] of every query to its own set (entries past N_s untouched, NaN);
    with packed_keys (pack_keys(keys)) the distance kernels read that copy."""
    ko = np.asarray(key_offsets_host if key_offsets_host is not None else key_offsets.cpu().numpy(), np.int64)
    qo = np.asarray(query_offsets_host if query_offsets_host is not None else query_offsets.cpu().numpy(), np.int64)
    B, d = queries.shape
    max_keys = int(np.diff(ko).max())
    max_q = int(np.diff(qo).max())
    ld = max_keys if ld is None else ld
    out = torch.full((B, ld), float("nan"), dtype=torch.float32, device=queries.device)
    code = _dtype_code(queries) | (KEYS_PACKED if packed_keys is not None else 0)
    src = keys if packed_keys is None else packed_keys
    st = load().knn_distances(_ptr(queries), _ptr(src), _ptr(key_sqnorms), _ptr(key_offsets), _ptr(query_offsets),
                              B, d, len(ko) - 1, max_keys, max_q, code, _ptr(out), ld, _stream(None))
    _lib.check("knn_distances", st)
    return out


def packed_keys_bytes(n: int, d: int, dtype: torch.dtype) -> int:
    """knn_packed_keys_bytes: bytes of the packed copy of n key rows of d elements (0: not packable)."""
    return int(load().knn_packed_keys_bytes(int(n), int(d), DTYPES[_TORCH_DTYPES[dtype]]))


def pack_keys(keys: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """knn_pack_keys: the packed copy of a [n, d] bf16/f16 key matrix (uint8 device tensor, into `out`
    when given), read by the matrix-core distance kernels in place of the row-major keys."""
    _need(keys.is_cuda and keys.is_contiguous() and keys.dim() == 2, "keys: contiguous 2-D device tensor")
    nbytes = packed_keys_bytes(keys.shape[0], keys.shape[1], keys.dtype) if keys.dtype in _TORCH_DTYPES else 0
    _need(nbytes > 0, "keys cannot be packed (bf16/f16 with d % 128 == 0 and d <= 65536)")
    if out is None:
        out = torch.empty(nbytes, dtype=torch.uint8, device=keys.device)
    _need(out.is_cuda and out.is_contiguous() and out.numel() * out.element_size() == nbytes,
          f"out: contiguous device tensor of {nbytes} bytes")
    st = load().knn_pack_keys(_ptr(keys), keys.shape[0], keys.shape[1], _dtype_code(keys), _ptr(out),
                              _stream(stream))
    _lib.check("knn_pack_keys", st)
    return out


def key_sqnorms(keys: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """knn_key_sqnorms: ||k||^2 per row, fp32, with the summation order knn_lm_mixture uses (into `out`
    when given: a contiguous [rows] fp32 device tensor)."""
    _need(keys.is_cuda and keys.is_contiguous() and keys.dim() == 2, "keys: contiguous 2-D device tensor")
    if out is None:
        out = torch.empty(keys.shape[0], dtype=torch.float32, device=keys.device)
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and out.numel() == keys.shape[0],
          "out: contiguous [rows] fp32 device tensor")
    st = load().knn_key_sqnorms(_ptr(keys), keys.shape[0], keys.shape[1], _dtype_code(keys), _ptr(out),
                                _stream(None))
    _lib.check("knn_key_sqnorms", st)
    return out


def mix(ids, dists, values, key_offsets, query_offsets, p_lm, mu, lam):
    """knn_mix: p_M [B, V] from caller-given neighbours (ids local to each query's set, squared distances)."""
    B, r = ids.shape
    V = p_lm.shape[1]
    S = key_offsets.numel() - 1
    out = torch.empty((B, V), dtype=torch.float32, device=p_lm.device)
    st = load().knn_mix(_ptr(ids), _ptr(dists), _ptr(values), _ptr(key_offsets), _ptr(query_offsets), _ptr(p_lm),
                        B, V, S, r, float(mu), float(lam), _ptr(out), _stream(None))
    _lib.check("knn_mix", st)
    return out


def mix_rrc(ids, dists, values, key_offsets, query_offsets, p_lm, mu, alpha, tau):
    """knn_mix_rrc: (p_M [B, V], lambda_t [B]) from caller-given neighbours with lambda_t
    from relative retrieval confidence."""
    B, r = ids.shape
    V = p_lm.shape[1]
    S = key_offsets.numel() - 1
    out = torch.empty((B, V), dtype=torch.float32, device=p_lm.device)
    lam = torch.empty(B, dtype=torch.float32, device=p_lm.device)
    st = load().knn_mix_rrc(_ptr(ids), _ptr(dists), _ptr(values), _ptr(key_offsets), _ptr(query_offsets),
                            _ptr(p_lm), B, V, S, r, float(mu), float(alpha), float(tau), _ptr(lam), _ptr(out),
                            _stream(None))
    _lib.check("knn_mix_rrc", st)
    return out, lam


def stream_read(buf: torch.Tensor, sink: torch.Tensor, stream=None):
    """knn_stream_read: one plain read of a contiguous device tensor (a measurement aid: the HBM
    read ceiling the distance stage is compared with); sink is a 1-element int32 device tensor."""
    _need(buf.is_cuda and buf.is_contiguous(), "buf: contiguous device tensor")
    _need(sink.is_cuda and sink.dtype == torch.int32 and sink.numel() >= 1, "sink: int32 device tensor")
    _lib.check("knn_stream_read", load().knn_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                                          _stream(stream)))


def mask_words(masked_rows, total_keys: int, device) -> torch.Tensor:
    """A key mask for knn_nest_step: int32 words with bit (i & 31) of word i >> 5 set for
    every masked global key row i (built on the host, then copied)."""
    words = np.zeros((total_keys + 31) // 32, dtype=np.uint32)
    rows = np.asarray(list(masked_rows), dtype=np.int64)
    if rows.size:
        _need(rows.min() >= 0 and rows.max() < total_keys, "masked row out of range")
        np.bitwise_or.at(words, rows >> 5, (np.uint32(1) << (rows & 31).astype(np.uint32)))
    return torch.as_tensor(words.view(np.int32), device=device)


def spec_verify(p_max, p_draft, next_token, draft_offsets, gamma, uniforms=None):
    """knn_spec_verify: (accepted count [n], replacement token or -1 [n]) per draft."""
    n = draft_offsets.numel() - 1
    dev = p_max.device
    n_acc = torch.empty(n, dtype=torch.int32, device=dev)
    tok = torch.empty(n, dtype=torch.int32, device=dev)
    st = load().knn_spec_verify(_ptr(p_max), _ptr(p_draft), _ptr(next_token), _ptr(draft_offsets), n, float(gamma),
                                _ptr(uniforms), _ptr(n_acc), _ptr(tok), _stream(None))
    _lib.check("knn_spec_verify", st)
    return n_acc, tok
